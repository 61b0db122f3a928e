/*
 * varrate.h -- C ABI of the variable-rank KV codec (VarRate, arXiv 2607.15498) for one
 * MI355X (gfx950) GPU.
 *
 * The codec compresses one layer's prompt KV cache (Algorithm 1) in three steps:
 *   1. salience   Sec. 3.2 Eq. (4): attention that the last w queries (the observation
 *                 window) pay each earlier token, averaged over the window and all query
 *                 heads, then the length-5 moving average;
 *   2. allocation Sec. 3.2 Eq. (5) + Sec. 3.1 Eq. (3): water-filling of the coded budget B
 *                 into one integer rank per token, floor r_min, cap R = d, sum = B exactly;
 *   3. projection Sec. 3.3 Eq. (6): each token's key and value are projected onto per-KV-head
 *                 orthonormal bases and truncated to the token's rank.
 * Decode (Sec. 4.4 "Cost" notes a fused kernel is what realises the saving) attends over
 * the compressed cache directly in rank space: the query is rotated into the key basis,
 * ragged coefficient rows are streamed, and the rank-space output is rotated back.
 *
 * Conventions for every entry point
 *   - All data pointers are DEVICE pointers (hipMalloc / torch CUDA tensors) owned by the
 *     caller unless stated otherwise; descriptors (varrate_shape, varrate_cache) are host
 *     structs.  Tensors are contiguous row-major, base addresses 16-byte aligned.
 *   - `stream` is a hipStream_t passed as void*; all device work is enqueued on it
 *     asynchronously.  No entry point synchronises the host or allocates device memory.
 *     The only state kept between calls is, per (kernel, device), the dynamic-LDS limit
 *     already raised with hipFuncSetAttribute (guarded by a lock, so calls from several
 *     host threads and on several devices are safe).
 *   - Arguments are validated synchronously before anything is enqueued; on error nothing
 *     is enqueued and a negative status is returned.  varrate_last_error() then returns a
 *     thread-local message.
 *   - Token notation: n = cached prompt tokens (window included), w = exact window = the
 *     observation window (last w tokens), N = n - w coded tokens, G KV heads, H query heads
 *     (H a multiple of G; query head h reads KV head h / (H/G)), d = 128 head dim.
 *   - dtype (VARRATE_BF16 or VARRATE_F32) is the storage type of K, V, window queries,
 *     decode queries, coefficients and decode outputs.  Bases are always fp32.
 *   - Workspaces are caller-allocated device buffers; their sizes come from the
 *     *_workspace_bytes functions.  A workspace must be zero-filled once before its first
 *     use; every call leaves it in that state again on completion (its counters reset
 *     themselves).  Calls that overlap in time on one workspace race.
 */
#ifndef VARRATE_H
#define VARRATE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define VARRATE_API __attribute__((visibility("default")))

/* ---- status codes -------------------------------------------------------------------- */
#define VARRATE_OK            0
#define VARRATE_EINVAL       -1   /* null pointer, bad shape/dtype, misaligned, small buffer */
#define VARRATE_EBUDGET      -2   /* N r_min > B, B > N R, or nothing to code (N <= 0)       */
#define VARRATE_EUNSUPPORTED -3   /* d != 128, H not a multiple of G, too many rows          */
#define VARRATE_EHIP         -4   /* a HIP launch or runtime call failed                      */

#define VARRATE_F32  0
#define VARRATE_BF16 1

#define VARRATE_HEAD_DIM 128   /* d = R: the bases are square, so full rank is exact        */
#define VARRATE_CHUNK    256   /* tokens per layout chunk (see varrate_cache)                */
#define VARRATE_COEF_PAD 64    /* extra elements after B in every coefficient stream         */
#define VARRATE_MAX_SEQS 64    /* sequences per varrate_decode_attn call                     */
#define VARRATE_MAX_QROWS 256  /* queries x heads-per-KV-head per sequence in one decode     */

/* One layer's problem statement (Algorithm 1 inputs). */
typedef struct varrate_shape {
    int64_t n;          /* cached prompt tokens, window included                            */
    int32_t G;          /* KV heads                                                         */
    int32_t H;          /* query heads (multiple of G)                                      */
    int32_t d;          /* head dim; must be 128                                            */
    int32_t w;          /* exact window = observation window, 1 <= w < n                    */
    int32_t r_min;      /* rank floor, 0 <= r_min <= 128                                    */
    int32_t kappa_pct;  /* KV budget kappa as an integer percent, 1..100                     */
    int32_t dtype;      /* VARRATE_BF16 or VARRATE_F32                                      */
    int32_t anchor_stride; /* 0: no anchors.  delta >= 2: the residual codec of Sec. 3.1 Eq. (2)
                              (bf16 layers): prefix tokens 0, delta, 2 delta, ... < n - w are
                              exact anchors, and every other prefix token is coded as its
                              residual to the mean of its 4 nearest anchors (see below)        */
    int32_t rope;       /* 0: position-free keys.  1: rotary keys (Sec. 3.1 "Joint per-token
                           vector", Algorithm 1 first and last steps): K, the window queries,
                           the decode queries and appended exact keys are post-RoPE, in the
                           rotate-half layout -- coordinates i and i + 64 form pair i, turned at
                           position p by the angle p * rope_theta[i] (radians; the exact product):
                               y_i = x_i cos - x_{i+64} sin,  y_{i+64} = x_i sin + x_{i+64} cos.
                           Prompt token t sits at position t.  The codec codes the un-rotated
                           keys (rotated back by -t, rounded to dtype, then projected), the
                           window rows stay exact and post-RoPE, and decode rebuilds each coded
                           key from its coefficients and rotates it to its position before the
                           score.  Not with anchors or quantised coefficients (EUNSUPPORTED).  */
    float   rope_theta[64]; /* per-pair frequencies (finite, >= 0; any scaling already applied) */
} varrate_shape;

/*
 * A compressed layer of one sequence.  The layout is part of the contract:
 *   - Coded tokens t in [0, N) are split into chunks of VARRATE_CHUNK consecutive tokens
 *     (the last chunk is ragged); n_chunks = ceil(N / VARRATE_CHUNK).
 *   - rank[t] (original order) is the integer rank of token t (Eq. 5, sum = B).
 *   - Inside chunk c the tokens are stored in order of (rank descending, index
 *     ascending); stored position i (global, i in [0, N)) holds token sidx[i] with rank
 *     srank[i].
 *   - Tile h of chunk c is its stored positions 16h .. 16h + 15 (positions past the chunk's
 *     end are absent, rank 0).  Its size m_h is the rank of its first position (the largest
 *     in the tile), and it takes 16 * m_h elements of every head stream at
 *         coef[g * coef_stride + chunk_off[c] + 16 * sum_{h' < h} m_h'],
 *     with chunk_off[c] = sum of 16 * m_h over the tiles of earlier chunks.  The K block is
 *     16 rows of m_h coordinates (row i: position 16h + i); the V block is m_h rows of 16
 *     positions (coordinate-major).  An entry (position, coordinate j) holds the position's
 *     projection onto basis row j (row j of P = j-th direction) when j < its rank, and 0
 *     otherwise.  Coefficients are stored in `dtype`.  chunk_off[n_chunks] <= B + 8 *
 *     VARRATE_CHUNK * n_chunks (a tile's size is bounded by the ranks of the tile before it).
 *   - k_exact/v_exact hold exact rows: slot e < w is token N + e (the window); slots
 *     e >= w are tokens appended after compression (varrate_append_exact).
 * Residual codec (shape->anchor_stride = delta > 0).  The prefix's na = ceil((n - w) / delta)
 * anchors (tokens a delta) are exact and the coded tokens are the other N = n - w - na prefix
 * tokens, numbered in order (coded token i is token i + i / (delta - 1) + 1); everything above
 * (ranks, storage order, tiles, budget) is over them, with B = floor(kappa n d / 100) -
 * (na + w) d (Eq. 3 with n_ref = na + w).  Each coded token's 4 nearest anchors are by
 * squared Euclidean distance over z_t = [k_t of all heads; v_t of all heads] (Eq. 2), computed
 * as ||z_a||^2 - 2 <z_a, z_t> with fp32 accumulation of exact bf16 products (ties to the
 * lower anchor); its stored coefficients are those of its residual x_t - (1/4) sum of the
 * anchors' rows (fp32, rounded to bf16 before the projection).
 * All pointers are device memory owned by the caller; sizes come from
 * varrate_cache_bytes().  n_exact is advanced on the host by varrate_compress (to w) and
 * varrate_append_exact.
 */
typedef struct varrate_cache {
    void*     coef_k;       /* [G][coef_stride] dtype                                      */
    void*     coef_v;       /* [G][coef_stride] dtype                                      */
    uint8_t*  rank;         /* [N], allocation padded to a multiple of 64 bytes             */
    uint8_t*  srank;        /* [N] ranks in stored order, allocation padded likewise        */
    uint32_t* sidx;         /* [N] stored position -> original token index                  */
    uint32_t* chunk_off;    /* [n_chunks + 1]                                               */
    void*     k_exact;      /* [G][cap][d] dtype                                            */
    void*     v_exact;      /* [G][cap][d] dtype                                            */
    int64_t   coef_stride;  /* elements per head stream, >= B + 2048 n_chunks + COEF_PAD    */
    int64_t   cap;          /* exact-slot capacity, >= w                                    */
    int64_t   n_exact;      /* exact slots in use                                           */
    int64_t   N;            /* coded tokens                                                 */
    int64_t   B;            /* coded budget (coefficients per head stream)                  */
    /* residual codec only (anchor_stride > 0; NULL / 0 otherwise):                          */
    void*     k_anchor;     /* [na][G][d] dtype: the anchors' keys, exact                   */
    void*     v_anchor;     /* [na][G][d] dtype: the anchors' values, exact                 */
    uint16_t* snn;          /* [N][4] the 4 nearest anchors (anchor numbers, nearest first)
                               of stored position i                                        */
    uint32_t* inv_off;      /* [na + 1] start of each anchor's list in inv_pos              */
    uint32_t* inv_pos;      /* [4 N] stored positions whose nearest anchors include anchor a,
                               at inv_pos[inv_off[a] .. inv_off[a + 1])                    */
    uint32_t* piece_off;    /* [na + 1] each anchor's list cut into pieces of 64 entries: the
                               pieces of anchor a are piece_off[a] .. piece_off[a + 1] - 1  */
    uint16_t* piece_anchor; /* [4 N / 64 + na] the anchor of each piece                     */
    int64_t   na;           /* anchors                                                      */
} varrate_cache;

/* Buffer sizes (bytes) a caller must allocate for one varrate_cache. */
typedef struct varrate_cache_bytes_t {
    int64_t N, B, n_chunks, coef_stride;
    size_t coef_k, coef_v, rank, srank, sidx, chunk_off, k_exact, v_exact;
    int64_t na;                                      /* residual codec: anchors (else 0)       */
    size_t k_anchor, v_anchor, snn, inv_off, inv_pos; /* residual codec buffers (else 0)       */
    size_t piece_off, piece_anchor;
} varrate_cache_bytes_t;

/* ---- diagnostics ---------------------------------------------------------------------- */
VARRATE_API const char* varrate_status_string(int status);
VARRATE_API const char* varrate_last_error(void);   /* thread-local text of the last failure           */
VARRATE_API int varrate_version(void);               /* ABI version (1)                                 */

/* Measurement aid (not part of the codec): reads `bytes` (a multiple of 16, > 0) of device
 * memory at `src` (16-byte aligned) with a plain streaming kernel of VARRATE_PROBE_WGS
 * workgroups, asynchronously on `stream`, so a caller can time what reading a given number of
 * bytes takes on this device.  `sink` is a device buffer of VARRATE_PROBE_WGS uint32 words that
 * the kernel may write (in practice it does not); its contents are meaningless.  EINVAL for
 * NULL or misaligned pointers or a bad size.                                                 */
#define VARRATE_PROBE_WGS 4096
VARRATE_API int varrate_read_probe(const void* src, size_t bytes, uint32_t* sink, void* stream);

/* ---- sizing ----------------------------------------------------------------------------- */
/* Coded budget of Sec. 3.1 Eq. (3) in per-head coefficient units, with kappa an integer
 * percent: B = floor(kappa_pct * n * d / 100) - w * d (the exact window costs w d).       */
VARRATE_API int64_t varrate_coded_budget(int64_t n, int32_t d, int32_t w, int32_t kappa_pct);

/* Validates the shape and budget feasibility (EBUDGET when N r_min > B or B > N d) and
 * fills the buffer sizes of one cache with exact capacity `cap` (>= w).                     */
VARRATE_API int varrate_cache_bytes(const varrate_shape* shape, int64_t cap, varrate_cache_bytes_t* out);

/* Workspace for varrate_salience / varrate_allocate / varrate_project / varrate_compress. */
VARRATE_API size_t varrate_compress_workspace_bytes(const varrate_shape* shape);
/* Workspace for varrate_decode_attn over S sequences of this shape with Q queries each. */
VARRATE_API size_t varrate_decode_workspace_bytes(const varrate_shape* shape, int32_t S, int32_t Q);

/* ---- stages ------------------------------------------------------------------------------ */
/* Sec. 3.2 Eq. (4) + length-5 moving average.
 * K: [n][G][d] dtype keys; Qw: [w][H][d] dtype observation-window queries (query i sits at
 * position n - w + i and attends causally to keys 0..n-w+i).  Writes sbar [N] fp32:
 *   s_t = (1/(w H)) sum_i sum_h softmax_t(<q_{i,h}, k_{t,g(h)}> / sqrt(d)),
 *   sbar_t = (s_{t-2} + ... + s_{t+2}) / 5 (out-of-range terms zero).                        */
VARRATE_API int varrate_salience(const varrate_shape* shape, const void* K, const void* Qw, float* sbar,
                     void* workspace, size_t workspace_bytes, void* stream);

/* Sec. 3.2 Eq. (5) water-filling on a given pooled salience sbar [N] fp32 (device).
 * Min-max normalisation to integer weights u_t = 1 + floor(2^24 (sbar_t - min)/(max - min))
 * (all equal when max == min), exact-integer water-filling with floor r_min and cap d, and
 * largest-remainder integer ranks (ties: larger u_t, then lower t) so that sum = B.
 * Writes cache->rank, the storage order cache->srank / cache->sidx (each chunk's tokens by
 * rank descending, index ascending) and cache->chunk_off; sets cache->N and cache->B.
 * Bit-exact and deterministic given sbar.                                                   */
VARRATE_API int varrate_allocate(const varrate_shape* shape, const float* sbar, varrate_cache* cache,
                     void* workspace, size_t workspace_bytes, void* stream);

/* Sec. 3.3 Eq. (6): projects K[0:N] and V[0:N] ([n][G][d] dtype) onto the bases
 * P_K, P_V ([G][d][d] fp32, row j = j-th direction, orthonormal rows) and keeps the leading
 * rank[t] coefficients of every token in the stored layout (needs cache->srank, cache->sidx
 * and cache->chunk_off from varrate_allocate).  Fills coef_k, coef_v, copies the window rows
 * K[N:n], V[N:n] into exact slots 0..w-1 and sets cache->n_exact = w.                       */
VARRATE_API int varrate_project(const varrate_shape* shape, const void* K, const void* V,
                    const float* P_K, const float* P_V, varrate_cache* cache,
                    void* workspace, size_t workspace_bytes, void* stream);

/* Algorithm 1 for one layer: the results of varrate_salience -> varrate_allocate ->
 * varrate_project, bit for bit (the pooling of the salience runs inside the allocation's
 * first pass, one launch fewer).  sbar_out ([N] fp32, device) receives the pooled salience
 * when non-NULL.  EINVAL for NULL inputs or inputs not 16-byte aligned.                      */
VARRATE_API int varrate_compress(const varrate_shape* shape, const void* K, const void* V, const void* Qw,
                     const float* P_K, const float* P_V, varrate_cache* cache, float* sbar_out,
                     void* workspace, size_t workspace_bytes, void* stream);

/* Appends one decode-time token (k_new, v_new: [G][d] dtype, device) to the exact slots
 * (tokens generated after compression stay exact).  EINVAL when the capacity is full.       */
VARRATE_API int varrate_append_exact(const varrate_shape* shape, varrate_cache* cache, const void* k_new,
                         const void* v_new, void* stream);

/* Residual codec stages (shape->anchor_stride > 0, bf16 layers).
 * varrate_anchor_search: the 4 nearest anchors of every coded token (coded order), nn
 *   [N][4] anchor numbers, nearest first; K, V [n][G][d].
 * varrate_anchor_encode: the rest of Algorithm 1 given the pooled salience of the whole
 *   prefix (sbar [n - w] fp32) and nn (from varrate_anchor_search or any other source, [N][4]
 *   coded order): the coded tokens' salience, the water-filling over them, residuals and their
 *   projection, the exact window and anchor rows, and the anchor lists of the cache.
 * varrate_compress on such a shape runs salience -> anchor search -> anchor encode.        */
VARRATE_API int varrate_anchor_search(const varrate_shape* shape, const void* K, const void* V, uint16_t* nn,
                          void* workspace, size_t workspace_bytes, void* stream);
VARRATE_API int varrate_anchor_encode(const varrate_shape* shape, const void* K, const void* V, const float* sbar,
                          const uint16_t* nn, const float* P_K, const float* P_V, varrate_cache* cache,
                          void* workspace, size_t workspace_bytes, void* stream);

/* Rank-space decode attention (the fused decode Sec. 4.4 calls for).
 * caches: host array of S compressed sequences of this shape (same layer, same bases).
 * q:   [S][Q][H][d] dtype decode queries (Q queries share each sequence's cache).
 * out: [S][Q][H][d] dtype.
 * For every sequence, query and head h (KV head g = h / (H/G)):
 *   q' = P_K[g] q / sqrt(d);  coded token t scores <q'[0:r_t], c^K_t>, exact slots score
 *   <q, k_e>/sqrt(d); softmax over all of them; out = P_V[g]^T (sum_t p_t c^V_t) +
 *   sum_e p_e v_e, which equals attention over the reconstructed cache of Eq. (6).
 * Constraints: S <= VARRATE_MAX_SEQS, Q * H / G <= VARRATE_MAX_QROWS.                       */
VARRATE_API int varrate_decode_attn(const varrate_shape* shape, const varrate_cache* caches, int32_t S,
                        const void* q, int32_t Q, const float* P_K, const float* P_V,
                        void* out, void* workspace, size_t workspace_bytes, void* stream);

/* ---- quantised coefficients (Sec. 3.3 "Composability") -------------------------------- */
/* The coefficients of a compressed bf16 layer quantised group-wise to b bits, the allocation
 * (ranks, storage order, exact rows) unchanged.  A group is one stored position's
 * coefficients of one head and stream in one 32-coordinate segment [32 s, 32 s + 32) below
 * its rank; symmetric absmax with Qmax = 2^(b-1) - 1:
 *     sc = binary16(fp32(amax / Qmax)),  k = clamp(rint(fp32(x / sc)), -Qmax, Qmax),
 * fp32 divisions correctly rounded, ties to even; a group with sc = 0 codes 0; x is the
 * stored bf16 coefficient, read back as k * sc.
 * Layout, per head stream (K and V alike), tile by tile in the layer's storage order: tile
 * h of chunk c (size m = its first position's rank, mq = m rounded up to a multiple of 8,
 * KS = ceil(m / 32)) takes 2 mq b + 32 KS bytes at
 *     code[g * q_stride + qchunk_off[c] + sum of the chunk's earlier tiles' bytes]:
 *   K: 16 rows of mq codes, code (position i, coordinate j) at bit b (i mq + j);
 *   V: mq rows of 16 codes, code (coordinate j, position i) at bit b (16 j + i);
 * then the KS x 16 binary16 scales of the tile, scale (group s, position i) at entry
 * 16 s + i.  Codes are two's complement b-bit fields packed from bit 0 of the tile upward;
 * codes past a position's rank, and of absent positions, are 0.                           */
typedef struct varrate_qcache {
    void*     code_k;      /* [G][q_stride] bytes                                           */
    void*     code_v;      /* [G][q_stride] bytes                                           */
    uint32_t* qchunk_off;  /* [n_chunks + 1] byte offset of each chunk in a head stream     */
    int64_t   q_stride;    /* bytes per head stream, a multiple of 16, >= varrate_qcache_bytes */
    int32_t   bits;        /* b: 3, 4 or 8                                                  */
    int32_t   reserved;
} varrate_qcache;

/* Bytes per head stream (q_stride) and of qchunk_off for b-bit codes of this shape's layer. */
VARRATE_API int varrate_qcache_bytes(const varrate_shape* shape, int32_t bits, int64_t* q_stride,
                         size_t* qchunk_off_bytes);

/* Quantises the coefficients of `cache` (filled by varrate_compress or varrate_project;
 * bf16 layers only) into `q` (q->bits, q->q_stride and the buffers set by the caller).
 * Two launches: the chunk offsets, then the codes and scales.  EINVAL for a bad q;
 * EUNSUPPORTED for fp32 layers or bits not in {3, 4, 8}.                                     */
VARRATE_API int varrate_quantize(const varrate_shape* shape, const varrate_cache* cache, varrate_qcache* q,
                     void* stream);

/* varrate_decode_attn over quantised coefficients: caches[s] supplies the storage order,
 * ranks and exact rows, qcaches[s] the codes of the same layer (all with the same bits
 * and q_stride).  Each coded token's score is sum over its groups of sc_K (q' . k) and its
 * value sum sc_V k, i.e. the reconstruct-in-place attention of Eq. (6) over the dequantised
 * coefficients.  Workspace as for varrate_decode_attn.                                      */
VARRATE_API int varrate_decode_attn_q(const varrate_shape* shape, const varrate_cache* caches,
                          const varrate_qcache* qcaches, int32_t S, const void* q, int32_t Q,
                          const float* P_K, const float* P_V, void* out, void* workspace,
                          size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): varrate_decode_attn without a workspace.
 * The partial records go to a fixed device array of VARRATE_DECODE_SCRATCH_BYTES that the
 * library holds on every device it runs on until the process ends (its address is looked
 * up once per device, on the first call there).  Same arguments, results and bits as
 * varrate_decode_attn; no allocation of any kind.  Returns VARRATE_EUNSUPPORTED when the
 * call needs more scratch than that (varrate_decode_scratch_need(); typically about
 * 4.3 MB: 512 partial records of 8320 bytes).  Every call on one device shares that
 * device's array: calls that overlap in time on one device (two streams, two host
 * threads) race and must be serialised by the caller.                                      */
#define VARRATE_DECODE_SCRATCH_BYTES (8u << 20)
VARRATE_API size_t varrate_decode_scratch_need(const varrate_shape* shape, int32_t S, int32_t Q);
VARRATE_API int varrate_decode_attn_noalloc(const varrate_shape* shape, const varrate_cache* caches, int32_t S,
                                const void* q, int32_t Q, const float* P_K, const float* P_V,
                                void* out, void* stream);

/* ---- shared cross-head basis ------------------------------------------------------------
 * Sec. 3.1 Eq. (1) "Joint per-token vector" and "Shared basis": every head's key and value of
 * a token form one vector z_t = [k_t of all G heads; v_t of all G heads] of Dz = 2 G d
 * entries, coded against ONE basis W in R^{R x Dz} (fp32, row j = j-th direction,
 * orthonormal rows; R a multiple of 128, 128 <= R <= min(1024, Dz)).  A coded token keeps
 * the leading r_t coefficients of c_t = W z_t (Eq. 6), one row for all heads and both K and
 * V, so a token at rank r costs r scalars and Eq. (3) reads B = floor(kappa n Dz / 100) -
 * w Dz, with ranks r_min <= r_t <= R (EBUDGET otherwise).  Salience, pooling and the exact
 * water-filling are those of the per-head codec (cap R instead of 128).  Position-free
 * keys, no anchors (shape->rope and shape->anchor_stride must be 0).
 * Layout (original token order): token t's coefficients are coef[offset[t] .. offset[t] +
 * rank[t]), offset = exclusive prefix sum of rank (offset[N] = B); chunk_off[c] = offset of
 * token 256 c.  Exact rows as in varrate_cache.  Decode: every query row (query x head) is
 * rotated into rank space once, q'_h = W_K,g q_h / sqrt(d) (W_K,g = the columns of head g's
 * keys), scored against the shared rows, and the rank-space value sums are rotated back by
 * W_V,g^T.  At most 32 query rows (Q H <= 32) per decode.                                    */
typedef struct varrate_jcache {
    void*     coef;         /* [coef_stride] dtype                                            */
    uint16_t* rank;         /* [N], allocation padded to a multiple of 64 bytes                */
    uint32_t* offset;       /* [N + 1]                                                        */
    uint32_t* chunk_off;    /* [n_chunks + 1]                                                 */
    void*     k_exact;      /* [G][cap][d] dtype                                              */
    void*     v_exact;      /* [G][cap][d] dtype                                              */
    int64_t   coef_stride;  /* elements, >= B + VARRATE_JOINT_PAD                             */
    int64_t   cap;          /* exact-slot capacity, >= w                                      */
    int64_t   n_exact;      /* exact slots in use                                             */
    int64_t   N;            /* coded tokens                                                   */
    int64_t   B;            /* coded budget in joint units                                    */
    int32_t   R;            /* basis rows                                                     */
    int32_t   reserved;
} varrate_jcache;
#define VARRATE_JOINT_PAD 2048  /* elements after B that decode may read (staging slack)      */

typedef struct varrate_jcache_bytes_t {
    int64_t N, B, n_chunks, coef_stride;
    size_t coef, rank, offset, chunk_off, k_exact, v_exact;
} varrate_jcache_bytes_t;

/* Sizes of one shared-basis cache with exact capacity cap (>= w); validates the shape and
 * the budget for R basis rows.                                                              */
VARRATE_API int varrate_jcache_bytes(const varrate_shape* shape, int32_t R, int64_t cap,
                                     varrate_jcache_bytes_t* out);
VARRATE_API size_t varrate_joint_compress_workspace_bytes(const varrate_shape* shape, int32_t R);
VARRATE_API size_t varrate_joint_decode_workspace_bytes(const varrate_shape* shape, int32_t R, int32_t S,
                                                        int32_t Q);
/* Algorithm 1 with the shared basis W [R][2 G d] (fp32): salience (sbar_out [N] when
 * non-NULL), water-filling of the joint budget with cap R, projection of z_t onto W truncated
 * to each rank.  Fills cache (R taken from cache->R) and copies the window rows.            */
VARRATE_API int varrate_joint_compress(const varrate_shape* shape, const void* K, const void* V, const void* Qw,
                                       const float* W, varrate_jcache* cache, float* sbar_out, void* workspace,
                                       size_t workspace_bytes, void* stream);
/* Decode attention over S shared-basis caches (same shape and R): q [S][Q][H][d] -> out
 * [S][Q][H][d], Q H <= 32.                                                                   */
VARRATE_API int varrate_joint_decode_attn(const varrate_shape* shape, const varrate_jcache* caches, int32_t S,
                                          const void* q, int32_t Q, const float* W, void* out, void* workspace,
                                          size_t workspace_bytes, void* stream);
/* varrate_append_exact for a shared-basis cache.                                             */
VARRATE_API int varrate_joint_append_exact(const varrate_shape* shape, varrate_jcache* cache, const void* k_new,
                                           const void* v_new, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* VARRATE_H */
