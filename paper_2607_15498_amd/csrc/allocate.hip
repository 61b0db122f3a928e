// Budgeted rank allocation (Sec. 3.2 Eq. (5), Algorithm 1 water-filling, integer ranks),
// exact integer arithmetic, plus the chunk-local storage order.
//
// Weights.  u_t = 1 + floor(2^24 (sbar_t - min) / (max - min)) with each fp64 operation
// rounded once (all equal when max == min), so the ranks are a function of the fp32 input.
//
// Water level.  With D = R - r_min, E = B - N r_min, the excess handed out at level
// lambda = D / tau is F(tau) = D (tau c_ge(tau) + s_lt(tau)) / tau, where c_ge counts
// u >= tau and s_lt sums u < tau.  F falls as tau grows, so the integer
//     tau_lo = max{ tau in [1, u_max] : D (tau c_ge(tau) + s_lt(tau)) >= E tau }
// is found from two histogram levels of u (12 + 12 bits) evaluated at bin edges.  The
// tokens capped at R are exactly {u > tau_lo} (ties exactly at R stay uncapped), k of them;
// the others get q_t = r_min + u_t M / Q with M = B - R k - r_min (N - k), Q = sum of their u.
// This is the fixed point of Algorithm 1's clip-and-redistribute loop.
//
// Integer ranks.  floor(q_t) plus one unit for the rho = B - sum floor(q_t) uncapped tokens
// with the largest keys (phi_t = (u_t M) mod Q, then u_t, then lower index), found by a
// most-significant-digit radix select (11-bit digits, common-prefix skipping) over the
// 2 x 64-bit key.  All arithmetic is integer: the ranks are bit-exact and deterministic.
//
// Kernel chain.  Every pass over the tokens is a grid of workgroups holding 1024 consecutive
// tokens each: 256 threads (wave w: the 256 tokens of one storage chunk, four coalesced loads
// per lane), or 1024 threads, one token each, in the passes that scan histograms (weights,
// fine, floors).  The small scans and searches between passes (4097 coarse bins, 4096 fine bins,
// 2048 digit bins, the threshold among the candidates) are repeated by every workgroup of the
// pass that needs them, which costs less than a launch of their own; workgroup 0 records the
// results for the later kernels.
//   al_minmax   per-workgroup min / max of sbar; clears the histograms and counters
//   al_weights  u, coarse histogram of u >> 12 (count, sum of the low bits), max u
//   al_fine     coarse scan -> the bin holding tau_lo; counts of the low bits inside it
//   al_floors   fine scan -> tau_lo, k, Q, M; floors, keys phi, sum of floors, histogram
//               of phi's top 11 significant bits
//   al_gather   rho; the digit bucket holding the rho-th largest key; its candidates
//   al_final    the exact threshold among the candidates; final ranks, each chunk's storage
//               order (srank, sidx) and its size in tile rectangles (16 x the largest rank of
//               each 16-position tile)
//   al_scan     (one workgroup; the allocation entry point only) chunk offsets.  In the
//               compress path the projection scans the chunk sizes itself.
#include "vr_internal.h"

namespace vr {

constexpr int AK_T = 256;                  // threads per workgroup of a token pass
constexpr int AK_PER = CHUNK / 64;         // tokens per lane (a wave holds one chunk)
constexpr int AK_TOK = AK_T * AK_PER;      // tokens per workgroup
constexpr int CBITS = 12;
constexpr int NCB = (1 << CBITS) + 1;      // coarse bins of u (u <= 2^24 + 1)
constexpr int NFB = 1 << CBITS;            // fine bins
constexpr int NDB = 2048;                  // selection digit bins (11 bits)
constexpr int SEL_CAP = 2048;              // candidates the selection finishes in LDS
constexpr uint64_t CAPPED = 1ull << 63;
constexpr int NRV = D + 1;                 // rank values 0..128
static_assert(AK_PER * 64 == CHUNK, "a wave holds one storage chunk");
static_assert(NFB % (4 * AK_T) == 0 && NDB % (4 * AK_T) == 0, "whole 16-byte staging loads per thread");

// Device-side state of one allocation (in the workspace, cleared by al_minmax).
struct AlCtl {
    unsigned long long fsum;     // sum of the floors (atomic)
    uint32_t umax;               // (atomic max)
    uint32_t ncand;              // gathered candidates (atomic)
    // water level (coarse: al_fine, fine: al_floors)
    int bbest, pad0;
    unsigned long long cge_next, slt_b;
    unsigned long long Q;
    long long M, kcap;
    uint32_t tau_lo;
    int sh0;                     // shift of the first selection digit
    // selection (al_gather, then every workgroup of al_final)
    unsigned long long pv, pm, T_hi, T_lo;
    long long need;              // rank of the threshold inside the bucket
    int done, any;
};

// Workspace: [coarse histogram | fine counts | digit counts | ctl] (the cleared region), then
// partial min/max, u, phi, candidates, chunk sizes.  A coarse bin packs its count (bits 40..63)
// and the sum of its tokens' low 12 bits (bits 0..39: at most 2^20 x 4095 < 2^40), so one
// 64-bit atomic adds both.
constexpr int CP_SHIFT = 40;
constexpr unsigned long long CP_LOW = (1ull << CP_SHIFT) - 1;
struct AlWs {
    unsigned long long* c_pack;
    uint32_t* f_cnt;
    uint32_t* d_cnt;
    AlCtl* ctl;
    uint32_t* clear;             // start of the cleared region, clear_words 32-bit words
    int clear_words;
    float2* mm;
    uint32_t* u;
    uint64_t* phi;
    uint64_t* cand;              // 2 x u64 per candidate (hi = phi, lo = (u, ~t))
    uint32_t* csum;              // each chunk's size (tile rectangles, or ranks for the shared basis)
};
constexpr int NCB_PAD = (NCB + 3) & ~3;

static AlWs al_ws(uint8_t* ws, int64_t N) {
    AlWs w;
    const int64_t nwg = (N + AK_TOK - 1) / AK_TOK;
    uint8_t* p = ws;
    w.clear = (uint32_t*)p;
    w.c_pack = (unsigned long long*)p; p += NCB_PAD * 8;
    w.f_cnt = (uint32_t*)p;           p += NFB * 4;
    w.d_cnt = (uint32_t*)p;           p += NDB * 4;
    w.ctl = (AlCtl*)p;                p += (sizeof(AlCtl) + 15) & ~(size_t)15;
    w.clear_words = (int)((p - ws) / 4);
    p = ws + align256(p - ws);
    w.mm = (float2*)p;                p += align256((size_t)nwg * sizeof(float2));
    w.u = (uint32_t*)p;               p += align256((size_t)N * 4);
    w.phi = (uint64_t*)p;             p += align256((size_t)N * 8);
    w.cand = (uint64_t*)p;            p += align256((size_t)N * 16);
    w.csum = (uint32_t*)p;
    return w;
}

size_t allocate_ws_bytes(const varrate_shape& sh) {
    const int64_t N = sh.n - sh.w;
    const int64_t nwg = (N + AK_TOK - 1) / AK_TOK;
    size_t b = align256(NCB_PAD * 8 + NFB * 4 + NDB * 4 + ((sizeof(AlCtl) + 15) & ~(size_t)15));
    b += align256((size_t)nwg * sizeof(float2)) + align256((size_t)N * 4) + align256((size_t)N * 8);
    const int64_t n_chunks = (N + CHUNK - 1) / CHUNK;
    return b + align256((size_t)N * 16) + align256((size_t)(n_chunks + 1) * 4);
}

// ---- workgroup primitives ----------------------------------------------------------------
template <typename T> __device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// Exclusive scan of one value per thread over NT threads; `tot` receives the total.
template <int NT, typename T>
__device__ T block_exscan(T v, T* wtot, T& tot) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    T x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        T y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    if (lane == 63) wtot[wid] = x;
    __syncthreads();
    T pre = 0, all = 0;
#pragma unroll
    for (int i = 0; i < NT / 64; ++i) {
        T wv = wtot[i];
        if (i < wid) pre += wv;
        all += wv;
    }
    __syncthreads();
    tot = all;
    return pre + x - v;
}

template <int NT, typename T, typename Op>
__device__ T block_reduce(T v, T* scratch, Op op) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = op(v, __shfl_xor(v, off, 64));
    if ((threadIdx.x & 63) == 0) scratch[threadIdx.x >> 6] = v;
    __syncthreads();
    T r = scratch[0];
#pragma unroll
    for (int i = 1; i < NT / 64; ++i) r = op(r, scratch[i]);
    __syncthreads();
    return r;
}

// In-place exclusive scan of n entries held in LDS; returns the total.
template <int NT, typename T>
__device__ T lds_exscan(T* a, int n, T* wtot) {
    const int per = (n + NT - 1) / NT;
    const int b = threadIdx.x * per;
    T loc = 0;
    for (int i = 0; i < per; ++i)
        if (b + i < n) loc += a[b + i];
    T tot;
    T pre = block_exscan<NT, T>(loc, wtot, tot);
    for (int i = 0; i < per; ++i)
        if (b + i < n) {
            T v = a[b + i];
            a[b + i] = pre;
            pre += v;
        }
    __syncthreads();
    return tot;
}

__device__ __forceinline__ uint64_t lo_key(uint32_t u, int64_t t) {
    return ((uint64_t)u << 24) | (uint64_t)(0xFFFFFFu - (uint32_t)t);
}

// Token of lane slot k in this workgroup: wave w holds tokens [256 w, 256 w + 256).
__device__ __forceinline__ int64_t al_tok(int k) {
    return (int64_t)blockIdx.x * AK_TOK + (threadIdx.x >> 6) * CHUNK + 64 * k + (threadIdx.x & 63);
}

// The u of one token (see the header); lo = min, range = max - min.
__device__ __forceinline__ uint32_t weight_of(float s, bool flat, double lo, double range) {
    if (flat) return (1u << 24) + 1u;
    const double num = (double)s - lo;
    double shat = num / range;
    // non-finite inputs cannot index past the histograms
    shat = shat >= 0.0 ? (shat <= 1.0 ? shat : 1.0) : 0.0;
    return 1u + (uint32_t)floor(shat * 16777216.0);
}

// ---- 1. min / max; clear the histograms and counters --------------------------------------
__global__ __launch_bounds__(AK_T) void al_minmax(const float* __restrict__ sbar, int64_t N,
                                                  float2* __restrict__ mm, uint32_t* __restrict__ clear,
                                                  int clear_words) {
    __shared__ float red[AK_T / 64];
    const int per = (clear_words + gridDim.x - 1) / gridDim.x;
    const int c0 = blockIdx.x * per, c1 = c0 + per < clear_words ? c0 + per : clear_words;
    for (int i = c0 + threadIdx.x; i < c1; i += AK_T) clear[i] = 0;
    float v[AK_PER];
#pragma unroll
    for (int k = 0; k < AK_PER; ++k) {
        const int64_t t = al_tok(k);
        v[k] = sbar[t < N ? t : N - 1];
    }
    float mn = v[0], mx = v[0];
#pragma unroll
    for (int k = 1; k < AK_PER; ++k) { mn = fminf(mn, v[k]); mx = fmaxf(mx, v[k]); }
    mn = block_reduce<AK_T>(mn, red, [](float a, float b) { return fminf(a, b); });
    mx = block_reduce<AK_T>(mx, red, [](float a, float b) { return fmaxf(a, b); });
    if (threadIdx.x == 0) mm[blockIdx.x] = make_float2(mn, mx);
}

// ---- 1'. (compress path) the same pass forming sbar from the salience column sums: the
//          pooled value of each of its tokens (the pooling kernel's arithmetic), written out
//          for the later passes, then min / max as above
__global__ __launch_bounds__(AK_T) void al_pool_minmax(const float* __restrict__ s_part, int64_t N, int G,
                                                       float inv_wh, float* __restrict__ sbar,
                                                       float2* __restrict__ mm, uint32_t* __restrict__ clear,
                                                       int clear_words) {
    __shared__ float red[AK_T / 64];
    __shared__ double sv[AK_TOK + 4];
    const int per = (clear_words + gridDim.x - 1) / gridDim.x;
    const int c0 = blockIdx.x * per, c1 = c0 + per < clear_words ? c0 + per : clear_words;
    for (int i = c0 + threadIdx.x; i < c1; i += AK_T) clear[i] = 0;
    const int64_t t0 = (int64_t)blockIdx.x * AK_TOK;
    // the column sums of every pooling term this thread forms, requested together
    constexpr int SV_IT = (AK_TOK + 4 + AK_T - 1) / AK_T;
    float part[SV_IT][POOL_MAXG];
#pragma unroll
    for (int it = 0; it < SV_IT; ++it) {
        const int64_t k = t0 - 2 + threadIdx.x + it * AK_T;
        pool_load(s_part, N, G, k >= 0 && k < N ? k : 0, part[it]);
    }
#pragma unroll
    for (int it = 0; it < SV_IT; ++it) {
        const int i = threadIdx.x + it * AK_T;
        const int64_t k = t0 - 2 + i;
        if (i < AK_TOK + 4) sv[i] = k >= 0 && k < N ? pool_sum(part[it], s_part, N, G, inv_wh, k) : 0.0;
    }
    __syncthreads();
    float v[AK_PER];
#pragma unroll
    for (int k = 0; k < AK_PER; ++k) {
        const int64_t t = al_tok(k);
        // tokens past N take token N - 1's value (inside this workgroup: t0 < N)
        v[k] = pool5(sv, (int)((t < N ? t : N - 1) - t0) + 2);
        if (t < N) sbar[t] = v[k];
    }
    float mn = v[0], mx = v[0];
#pragma unroll
    for (int k = 1; k < AK_PER; ++k) { mn = fminf(mn, v[k]); mx = fmaxf(mx, v[k]); }
    mn = block_reduce<AK_T>(mn, red, [](float a, float b) { return fminf(a, b); });
    mx = block_reduce<AK_T>(mx, red, [](float a, float b) { return fmaxf(a, b); });
    if (threadIdx.x == 0) mm[blockIdx.x] = make_float2(mn, mx);
}

// The histogram passes run 1024 threads, one token each (the same 1024 tokens per workgroup
// as the other passes): their per-thread scans over the bins are then 4 to 5 bins long, with
// four waves per SIMD to hide each other's latency.
constexpr int AW_T = AK_TOK;
__device__ __forceinline__ int64_t aw_tok() { return (int64_t)blockIdx.x * AK_TOK + threadIdx.x; }

// Global min / max from the per-workgroup partials (exact, so any order gives the same).
template <int NT>
__device__ __forceinline__ float2 al_range(const float2* __restrict__ mm, int nwg, float* red) {
    float mn = INFINITY, mx = -INFINITY;
    for (int i = threadIdx.x; i < nwg; i += NT) {
        const float2 p = mm[i];
        mn = fminf(mn, p.x);
        mx = fmaxf(mx, p.y);
    }
    mn = block_reduce<NT>(mn, red, [](float a, float b) { return fminf(a, b); });
    mx = block_reduce<NT>(mx, red, [](float a, float b) { return fmaxf(a, b); });
    return make_float2(mn, mx);
}

// ---- 2. weights and the coarse histogram ----------------------------------------------------
__global__ __launch_bounds__(AW_T) void al_weights(const float* __restrict__ sbar, int64_t N,
                                                   const float2* __restrict__ mm, int nwg,
                                                   uint32_t* __restrict__ u_ws,
                                                   unsigned long long* __restrict__ c_pack,
                                                   AlCtl* __restrict__ ctl) {
    __shared__ uint32_t cnt[NCB_PAD], low[NCB_PAD];
    __shared__ float red[AW_T / 64];
    __shared__ uint32_t redu[AW_T / 64];
    const int64_t t = aw_tok();
    const float s = sbar[t < N ? t : N - 1];
    for (int i = threadIdx.x; i < NCB_PAD; i += AW_T) { cnt[i] = 0; low[i] = 0; }
    const float2 r = al_range<AW_T>(mm, nwg, red);     // (its barriers also order the clearing)
    const bool flat = !(r.y > r.x);
    const double lo = (double)r.x, range = (double)r.y - lo;
    uint32_t umax = 0;
    if (t < N) {
        const uint32_t u = weight_of(s, flat, lo, range);
        u_ws[t] = u;
        umax = u;
        atomicAdd(&cnt[u >> CBITS], 1u);
        atomicAdd(&low[u >> CBITS], u & ((1u << CBITS) - 1));
    }
    umax = block_reduce<AW_T>(umax, redu, [](uint32_t a, uint32_t b) { return a > b ? a : b; });
    if (threadIdx.x == 0) atomicMax(&ctl->umax, umax);
    for (int i = threadIdx.x; i < NCB; i += AW_T) {
        const uint32_t c = cnt[i];
        if (c) atomicAdd(&c_pack[i], ((unsigned long long)c << CP_SHIFT) | low[i]);
    }
}

// ---- 3. coarse level; fine histogram ----------------------------------------------------------
// Thread i holds bins [CPT i, CPT i + CPT) of a scan in registers.
constexpr int CPT = (NCB + AW_T - 1) / AW_T;    // 5 coarse bins per thread
constexpr int FPT = NFB / AW_T;                 // 4 fine bins per thread
static_assert(FPT == 4, "one 16-byte load of fine counts per thread");

__global__ __launch_bounds__(AW_T) void al_fine(int64_t N, int64_t B, int r_min, int R,
                                                const uint32_t* __restrict__ u_ws,
                                                const unsigned long long* __restrict__ c_pack,
                                                uint32_t* __restrict__ f_cnt, AlCtl* __restrict__ ctl) {
    // the coarse histogram staged through LDS with coalesced loads, then the fine counts
    __shared__ union {
        unsigned long long bins[CPT * AW_T];
        uint32_t cnt[NFB];
    } sm;
    uint32_t* cnt = sm.cnt;
    __shared__ uint32_t wt32[AW_T / 64];
    __shared__ unsigned long long wt64[AW_T / 64];
    __shared__ unsigned long long s_edge[2];
    const int64_t t = aw_tok();
    const uint32_t u = u_ws[t < N ? t : N - 1];
    {
        unsigned long long st[CPT];
#pragma unroll
        for (int j = 0; j < CPT; ++j) {
            const int i = threadIdx.x + j * AW_T;
            st[j] = c_pack[i < NCB ? i : NCB - 1];
        }
#pragma unroll
        for (int j = 0; j < CPT; ++j) sm.bins[threadIdx.x + j * AW_T] = st[j];
    }
    __syncthreads();
    const int b0 = CPT * threadIdx.x;
    const uint32_t umax = ctl->umax;
    const int nb = (int)(umax >> CBITS) + 1;
    // bin sums and this thread's totals (bins >= nb are empty: u <= umax; bins past NCB too)
    uint32_t c[CPT];
    unsigned long long l[CPT];
    uint32_t lc = 0;
    unsigned long long ls = 0;
#pragma unroll
    for (int j = 0; j < CPT; ++j) {
        const int b = b0 + j;
        const unsigned long long v = sm.bins[b];
        c[j] = b < nb ? (uint32_t)(v >> CP_SHIFT) : 0u;
        l[j] = b < nb ? (v & CP_LOW) + (unsigned long long)c[j] * ((uint64_t)b << CBITS) : 0ull;   // sum of u in bin b
        lc += c[j];
        ls += l[j];
    }
    uint32_t tc;
    unsigned long long ts;
    uint32_t pc = block_exscan<AW_T, uint32_t>(lc, wt32, tc);
    // (every thread has its bins in registers: the staging area becomes the fine counts)
    for (int i = threadIdx.x; i < NFB; i += AW_T) cnt[i] = 0;
    unsigned long long ps = block_exscan<AW_T, unsigned long long>(ls, wt64, ts);
    const uint64_t Dr = (uint64_t)(R - r_min);
    const uint64_t E = (uint64_t)(B - N * (int64_t)r_min);
    // the predicate at coarse edges tau_b = max(1, b << 12): c_ge = N - cnt_ex[b], s_lt = sm_ex[b]
    int bbest = 0;
    {
        uint32_t rc = pc;
        unsigned long long rs = ps;
#pragma unroll
        for (int j = 0; j < CPT; ++j) {
            const int b = b0 + j;
            const uint64_t tau = b == 0 ? 1 : ((uint64_t)b << CBITS);
            const uint64_t cge = (uint64_t)N - rc;
            if (b < nb && Dr * (tau * cge + rs) >= E * tau) bbest = b;
            rc += c[j];
            rs += l[j];
        }
    }
    bbest = (int)block_reduce<AW_T, uint32_t>((uint32_t)bbest, wt32,
                                              [](uint32_t a, uint32_t b) { return a > b ? a : b; });
    {
        uint32_t rc = pc;
        unsigned long long rs = ps;
#pragma unroll
        for (int j = 0; j < CPT; ++j) {
            if (b0 + j == bbest) {
                s_edge[0] = (uint64_t)N - (rc + c[j]);   // tokens in bins above bbest
                s_edge[1] = rs;                          // sum of u in bins below bbest
            }
            rc += c[j];
            rs += l[j];
        }
    }
    __syncthreads();
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        ctl->bbest = bbest;
        ctl->cge_next = s_edge[0];
        ctl->slt_b = s_edge[1];
    }
    // fine counts of the low 12 bits inside bin bbest (every u there is (bbest << 12) + f)
    if (t < N && (int)(u >> CBITS) == bbest) atomicAdd(&cnt[u & (NFB - 1)], 1u);
    __syncthreads();
    for (int i = threadIdx.x; i < NFB; i += AW_T) {
        const uint32_t cc = cnt[i];
        if (cc) atomicAdd(&f_cnt[i], cc);
    }
}

// ---- 4. fine level; floors, keys and the first selection digit --------------------------------
// RT: the rank type, uint8_t (per-head codec, R = 128) or uint16_t (shared basis, R <= 1024)
template <typename RT>
__global__ __launch_bounds__(AW_T) void al_floors(int64_t N, int64_t B, int r_min, int R,
                                                  const uint32_t* __restrict__ u_ws,
                                                  const uint32_t* __restrict__ f_cnt,
                                                  RT* __restrict__ rank, uint64_t* __restrict__ phi_ws,
                                                  uint32_t* __restrict__ d_cnt, AlCtl* __restrict__ ctl) {
    __shared__ uint32_t cnt[NDB];
    __shared__ uint32_t wt32[AW_T / 64];
    __shared__ unsigned long long wt64[AW_T / 64];
    __shared__ unsigned long long s_edge[2];
    const int64_t t = aw_tok();
    const uint32_t u = u_ws[t < N ? t : N - 1];
    const int f0 = FPT * threadIdx.x;
    uint32_t c[FPT];
    {
        const uint4 v = reinterpret_cast<const uint4*>(f_cnt)[threadIdx.x];
        c[0] = v.x; c[1] = v.y; c[2] = v.z; c[3] = v.w;
    }
    for (int i = threadIdx.x; i < NDB; i += AW_T) cnt[i] = 0;
    const uint32_t umax = ctl->umax;
    const int bbest = ctl->bbest;
    const uint64_t cge_next = ctl->cge_next, slt_b = ctl->slt_b;
    const uint64_t base_tau = (uint64_t)bbest << CBITS;
    uint32_t lc = 0;
    unsigned long long ls = 0;
#pragma unroll
    for (int j = 0; j < FPT; ++j) {
        lc += c[j];
        ls += (unsigned long long)c[j] * (base_tau + (uint64_t)(f0 + j));
    }
    uint32_t tc;
    unsigned long long ts;
    const uint32_t pc = block_exscan<AW_T, uint32_t>(lc, wt32, tc);
    const unsigned long long ps = block_exscan<AW_T, unsigned long long>(ls, wt64, ts);
    const uint64_t Dr = (uint64_t)(R - r_min);
    const uint64_t E = (uint64_t)(B - N * (int64_t)r_min);
    const uint64_t fc_total = tc;
    const int f_lo = bbest == 0 ? 1 : 0;
    const int f_hi = (int)(((uint64_t)umax - base_tau) < (uint64_t)(NFB - 1) ? (umax - base_tau) : (NFB - 1));
    int fbest = f_lo;
    {
        uint32_t rc = pc;
        unsigned long long rs = ps;
#pragma unroll
        for (int j = 0; j < FPT; ++j) {
            const int f = f0 + j;
            const uint64_t tau = base_tau + f;
            const uint64_t cge = cge_next + fc_total - rc;
            const uint64_t slt = slt_b + rs;
            if (f >= f_lo && f <= f_hi && Dr * (tau * cge + slt) >= E * tau) fbest = f;
            rc += c[j];
            rs += (unsigned long long)c[j] * (base_tau + (uint64_t)f);
        }
    }
    fbest = (int)block_reduce<AW_T, uint32_t>((uint32_t)fbest, wt32,
                                              [](uint32_t a, uint32_t b) { return a > b ? a : b; });
    {
        uint32_t rc = pc;
        unsigned long long rs = ps;
#pragma unroll
        for (int j = 0; j < FPT; ++j) {
            rc += c[j];
            rs += (unsigned long long)c[j] * (base_tau + (uint64_t)(f0 + j));
            if (f0 + j == fbest) { s_edge[0] = rc; s_edge[1] = rs; }   // inclusive of fbest
        }
    }
    __syncthreads();
    const uint32_t tau_lo = (uint32_t)(base_tau + fbest);
    const int64_t kcap = (int64_t)(cge_next + fc_total - s_edge[0]);
    const uint64_t Q = slt_b + s_edge[1];
    const int64_t M = B - (int64_t)R * kcap - (int64_t)r_min * (N - kcap);
    const double invQ = 1.0 / (double)Q;
    // first selection digit: phi < Q, so its top 11 significant bits need no range pass
    const uint64_t qm1 = Q > 1 ? Q - 1 : 1;
    const int qb = 64 - __clzll((long long)qm1);
    const int sh0 = qb > 11 ? qb - 11 : 0;
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        ctl->tau_lo = tau_lo;
        ctl->kcap = kcap;
        ctl->Q = Q;
        ctl->M = M;
        ctl->sh0 = sh0;
    }

    unsigned long long fsum = 0;
    if (t < N) {
        uint32_t base;
        uint64_t phi;
        if (u > tau_lo) {
            base = (uint32_t)R;
            phi = CAPPED;
        } else {
            // num < 2^52 and Q < 2^45 are exact in fp64; the reciprocal quotient is within
            // one unit of floor(num / Q) and the integer remainder corrects it exactly
            const uint64_t num = (uint64_t)u * (uint64_t)M;
            int64_t f = (int64_t)((double)num * invQ);
            int64_t rem = (int64_t)num - f * (int64_t)Q;
            if (rem < 0) { f -= 1; rem += (int64_t)Q; }
            if (rem >= (int64_t)Q) { f += 1; rem -= (int64_t)Q; }
            phi = (uint64_t)rem;
            base = (uint32_t)(r_min + f);
            atomicAdd(&cnt[(phi >> sh0) & (NDB - 1)], 1u);
        }
        rank[t] = (RT)base;
        phi_ws[t] = phi;
        fsum = base;
    }
    fsum = block_reduce<AW_T, unsigned long long>(fsum, wt64,
                                                  [](unsigned long long a, unsigned long long b) { return a + b; });
    if (threadIdx.x == 0) atomicAdd(&ctl->fsum, fsum);
    for (int i = threadIdx.x; i < NDB; i += AW_T) {
        const uint32_t c = cnt[i];
        if (c) atomicAdd(&d_cnt[i], c);
    }
}

// ---- 5. selection ------------------------------------------------------------------------------
struct SelState {
    uint64_t pv, pm;   // fixed prefix value / mask of the field being narrowed
    uint64_t T_hi, T_lo;
    int64_t need;
    int phase;         // 0: narrowing phi, 1: narrowing (u, ~t)
    int done;
};

// Most-significant-digit narrowing of the threshold over the candidates enumerated by
// visit(f) (f(hi, lo) per candidate) by NT threads, starting from `sel`.
template <int NT, class Visit>
__device__ void radix_narrow(Visit visit, SelState& sel, uint32_t* cnt, uint32_t* wtot32,
                             unsigned long long* wtot64) {
    constexpr int DPT = NDB / NT;       // digits per thread, in descending order
    const int tid = threadIdx.x;
    // every round fixes at least one more bit of the field or ends the phase, so two 64-bit
    // fields finish within 2 * 65 rounds; the bound only guards against a broken invariant
    for (int round = 0; round < 2 * 65 && !sel.done; ++round) {
        const int phase = sel.phase;
        const uint64_t pv = sel.pv, pm = sel.pm, T_hi = sel.T_hi;
        auto field = [&](uint64_t hi, uint64_t lo, uint64_t& f) -> bool {
            if (phase == 0) {
                f = hi;
            } else {
                if (hi != T_hi) return false;
                f = lo;
            }
            return (f & pm) == pv;
        };
        uint64_t fmn = ~0ull, fmx = 0;
        visit([&](uint64_t hi, uint64_t lo) {
            uint64_t f;
            if (field(hi, lo, f)) {
                fmn = f < fmn ? f : fmn;
                fmx = f > fmx ? f : fmx;
            }
        });
        fmn = block_reduce<NT, unsigned long long>(fmn, wtot64, [](unsigned long long a, unsigned long long b) { return a < b ? a : b; });
        fmx = block_reduce<NT, unsigned long long>(fmx, wtot64, [](unsigned long long a, unsigned long long b) { return a > b ? a : b; });
        if (fmn == fmx) {
            if (tid == 0) {
                if (phase == 0) {
                    sel.T_hi = fmn; sel.phase = 1; sel.pv = 0; sel.pm = 0;
                } else {
                    sel.T_lo = fmn; sel.done = 1;   // keys are unique: a single candidate
                }
            }
            __syncthreads();
            continue;
        }
        const int p = 63 - __clzll((long long)(fmn ^ fmx));
        const int sh = p > 10 ? p - 10 : 0;
        const uint64_t dmask = (1ull << (p - sh + 1)) - 1;
        const uint64_t above_mask = (p == 63) ? 0ull : ~((2ull << p) - 1);
        for (int i = tid; i < NDB; i += NT) cnt[i] = 0;
        __syncthreads();
        visit([&](uint64_t hi, uint64_t lo) {
            uint64_t f;
            if (field(hi, lo, f)) atomicAdd(&cnt[(f >> sh) & dmask], 1u);
        });
        __syncthreads();
        uint32_t c[DPT], loc = 0;
#pragma unroll
        for (int j = 0; j < DPT; ++j) { c[j] = cnt[NDB - 1 - DPT * tid - j]; loc += c[j]; }
        uint32_t tot;
        uint32_t above = block_exscan<NT, uint32_t>(loc, wtot32, tot);
        const int64_t need = sel.need;
        __syncthreads();                          // every thread has read sel before it changes
#pragma unroll
        for (int j = 0; j < DPT; ++j) {
            if ((int64_t)above < need && need <= (int64_t)(above + c[j])) {
                const int hit = NDB - 1 - DPT * tid - j;
                const int64_t nn = need - (int64_t)above;
                const uint64_t npv = (fmn & above_mask) | ((uint64_t)hit << sh);
                sel.need = nn;
                sel.pv = npv;
                sel.pm = ~((1ull << sh) - 1);
                if ((int64_t)c[j] == nn) {
                    if (phase == 0) { sel.T_hi = npv; sel.T_lo = 0; }
                    else { sel.T_lo = npv; }
                    sel.done = 1;
                }
            }
            above += c[j];
        }
        __syncthreads();
    }
}

// The digit bucket holding the rho-th largest key (every workgroup), and its candidates
// into a list.
__global__ __launch_bounds__(AK_T) void al_gather(int64_t N, int64_t B, const uint32_t* __restrict__ u_ws,
                                                  const uint64_t* __restrict__ phi_ws,
                                                  const uint32_t* __restrict__ d_cnt,
                                                  uint64_t* __restrict__ cand, AlCtl* __restrict__ ctl) {
    __shared__ uint32_t wt32[AK_T / 64];
    __shared__ int s_hit;
    __shared__ uint32_t s_above, s_hcnt, s_n, s_base;
    __shared__ uint4 sd[NDB / 4];                 // the digit counts (coalesced loads)
    uint64_t phi[AK_PER];
    uint32_t u[AK_PER];
#pragma unroll
    for (int k = 0; k < AK_PER; ++k) {
        const int64_t t = al_tok(k);
        phi[k] = phi_ws[t < N ? t : N - 1];
        u[k] = u_ws[t < N ? t : N - 1];
    }
    const int64_t rho = B - (int64_t)ctl->fsum;
    const int sh0 = ctl->sh0;
    if (threadIdx.x == 0) { s_hit = -1; s_n = 0; }
    // descending digit order: thread i holds digits 2047 - 8 i .. 2040 - 8 i
    constexpr int DPT = NDB / AK_T;
    {
        constexpr int DL = NDB / 4 / AK_T;
        uint4 st[DL];
#pragma unroll
        for (int j = 0; j < DL; ++j) st[j] = reinterpret_cast<const uint4*>(d_cnt)[threadIdx.x + j * AK_T];
#pragma unroll
        for (int j = 0; j < DL; ++j) sd[threadIdx.x + j * AK_T] = st[j];
    }
    __syncthreads();
    const uint32_t* sdc = reinterpret_cast<const uint32_t*>(sd);
    uint32_t c[DPT], loc = 0;
#pragma unroll
    for (int j = 0; j < DPT; ++j) { c[j] = sdc[NDB - 1 - DPT * threadIdx.x - j]; loc += c[j]; }
    uint32_t tot;
    uint32_t above = block_exscan<AK_T, uint32_t>(loc, wt32, tot);
    if (rho > 0) {
#pragma unroll
        for (int j = 0; j < DPT; ++j) {
            if ((int64_t)above < rho && rho <= (int64_t)(above + c[j])) {
                s_hit = NDB - 1 - DPT * threadIdx.x - j;
                s_above = above;
                s_hcnt = c[j];
            }
            above += c[j];
        }
    }
    __syncthreads();
    const int hit = s_hit;
    // rho <= 0 selects nothing; rho > 0 always lands in a bucket (rho < uncapped count)
    const int64_t need = hit < 0 ? 0 : rho - (int64_t)s_above;
    const bool done0 = hit < 0 || (int64_t)s_hcnt == need;
    const uint64_t pv = hit < 0 ? 0 : (uint64_t)hit << sh0;
    const uint64_t pm = ~((1ull << sh0) - 1);
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        ctl->any = rho > 0 && hit >= 0;
        ctl->T_hi = hit < 0 ? ~0ull : pv;      // the whole bucket is taken when done here
        ctl->T_lo = 0;
        ctl->pv = pv;
        ctl->pm = pm;
        ctl->need = need;
        ctl->done = done0;
    }
    if (done0) return;                         // (the same in every workgroup)
    // candidates of the bucket: a workgroup-local slot first, then one global reservation
    uint32_t slot[AK_PER];
    bool mine[AK_PER];
#pragma unroll
    for (int k = 0; k < AK_PER; ++k) {
        mine[k] = al_tok(k) < N && phi[k] != CAPPED && (phi[k] & pm) == pv;
        if (mine[k]) slot[k] = atomicAdd(&s_n, 1u);
    }
    __syncthreads();
    if (threadIdx.x == 0 && s_n) s_base = atomicAdd(&ctl->ncand, s_n);
    __syncthreads();
#pragma unroll
    for (int k = 0; k < AK_PER; ++k)
        if (mine[k]) {
            const uint64_t i = (uint64_t)(s_base + slot[k]);
            cand[2 * i] = phi[k];
            cand[2 * i + 1] = lo_key(u[k], al_tok(k));
        }

}

// The exact threshold among the bucket's candidates, found by every workgroup of the final
// pass from the same list with the same arithmetic, so all of them agree and no one-workgroup
// pass sits between the gather and the final ranks.  Up to AK_T candidates (the usual case: a
// digit bucket holds about 2^-11 of the uncapped tokens) rank one another directly, each
// candidate's comparisons split over the workgroup; up to SEL_CAP go through the radix
// narrowing in LDS; more (many equal weights) through the same narrowing over the list in
// memory.
struct AlSelSmem {
    unsigned long long chi[SEL_CAP], clo[SEL_CAP];
    uint32_t cnt[NDB];
    unsigned long long wt64[AK_T / 64];
    uint32_t wt32[AK_T / 64];
    unsigned long long T[2];
    SelState sel;
};

// (my_hi, my_lo): list entry min(threadIdx.x, N - 1), loaded by the caller ahead of time
__device__ void al_threshold(int64_t N, const uint64_t* __restrict__ cand, const AlCtl* __restrict__ ctl,
                             uint64_t my_hi, uint64_t my_lo, AlSelSmem& s, uint64_t& T_hi, uint64_t& T_lo) {
    const int tid = threadIdx.x;
    if (ctl->done) {                 // nothing to take (T = ~0), or the whole bucket (T = its edge)
        T_hi = ctl->T_hi;
        T_lo = ctl->T_lo;
        return;
    }
    const int nc = (int)ctl->ncand;
    const int64_t need = ctl->need;
    if (nc <= AK_T) {
        if (tid < nc) { s.chi[tid] = my_hi; s.clo[tid] = my_lo; s.cnt[tid] = 0; }
        __syncthreads();
        // candidate i = tid mod nc against slice tid / nc of the list (nseg slices)
        const int nseg = AK_T / nc, per = (nc + nseg - 1) / nseg;
        if (tid < nc * nseg) {
            const int i = tid % nc, j0 = (tid / nc) * per;
            const int j1 = j0 + per < nc ? j0 + per : nc;
            const uint64_t h = s.chi[i], l = s.clo[i];
            uint32_t above = 0;
            for (int j = j0; j < j1; ++j) {
                const uint64_t hj = s.chi[j], lj = s.clo[j];
                above += (hj > h || (hj == h && lj > l)) ? 1u : 0u;
            }
            if (above) atomicAdd(&s.cnt[i], above);
        }
        __syncthreads();
        // keys are unique: exactly one candidate has need - 1 larger ones
        if (tid < nc && (int64_t)s.cnt[tid] == need - 1) { s.T[0] = s.chi[tid]; s.T[1] = s.clo[tid]; }
        __syncthreads();
        T_hi = s.T[0];
        T_lo = s.T[1];
        return;
    }
    if (tid == 0) {
        s.sel.pv = ctl->pv; s.sel.pm = ctl->pm; s.sel.need = need;
        s.sel.T_hi = ~0ull; s.sel.T_lo = ~0ull; s.sel.phase = 0; s.sel.done = 0;
    }
    if (nc <= SEL_CAP) {
        for (int i = tid; i < nc; i += AK_T) { s.chi[i] = cand[2 * i]; s.clo[i] = cand[2 * i + 1]; }
        __syncthreads();
        radix_narrow<AK_T>([&](auto f) {
            for (int i = tid; i < nc; i += AK_T) f(s.chi[i], s.clo[i]);
        }, s.sel, s.cnt, s.wt32, s.wt64);
    } else {
        __syncthreads();
        // sixteen entries per thread in flight at a time (clamped addresses, masked entries)
        radix_narrow<AK_T>([&](auto f) {
            constexpr int BT = 16;
            for (int i0 = 0; i0 < nc; i0 += BT * AK_T) {
                uint64_t h[BT], l[BT];
#pragma unroll
                for (int k = 0; k < BT; ++k) {
                    const int i = i0 + k * AK_T + tid;
                    const int ii = i < nc ? i : 0;
                    h[k] = cand[2 * ii];
                    l[k] = cand[2 * ii + 1];
                }
#pragma unroll
                for (int k = 0; k < BT; ++k)
                    if (i0 + k * AK_T + tid < nc) f(h[k], l[k]);
            }
        }, s.sel, s.cnt, s.wt32, s.wt64);
    }
    T_hi = s.sel.T_hi;
    T_lo = s.sel.T_lo;
}

// Stored order of one chunk per wave: rank descending, token index ascending (a stable
// counting sort).  Lane `lane` holds the ranks r[k] of tokens t0 + 64 k + lane (tokens past N
// take no part); token lane + 64 k is bit `lane` of word k of its rank's mask, so a token's
// place is (#tokens of higher rank) + (#earlier tokens of its rank).  Writes srank / sidx at
// the chunk's positions and returns the chunk's size in tile rectangles (16 x the first,
// largest rank of each 16-position tile), summed over the wave.  m and above are the wave's
// own LDS scratch; the function holds workgroup barriers, so every wave calls it together.
__device__ uint32_t chunk_order(unsigned long long (*m)[4], uint16_t* above, const uint32_t (&r)[AK_PER],
                                int64_t t0, int64_t N, uint8_t* __restrict__ srank,
                                uint32_t* __restrict__ sidx) {
    const int lane = threadIdx.x & 63;
    for (int i = lane; i < NRV * 4; i += 64) (&m[0][0])[i] = 0ull;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < AK_PER; ++k)
        if (t0 + 64 * k + lane < N) atomicOr(&m[r[k]][k], 1ull << lane);
    __syncthreads();
    {
        // lane covers rank values 128 - 3 lane - e (descending), then a wave exclusive scan
        uint32_t h[3], loc = 0;
#pragma unroll
        for (int e = 0; e < 3; ++e) {
            const int q = 3 * lane + e;
            h[e] = 0;
            if (q < NRV) {
                const unsigned long long* mm = m[NRV - 1 - q];
                h[e] = __popcll(mm[0]) + __popcll(mm[1]) + __popcll(mm[2]) + __popcll(mm[3]);
            }
            loc += h[e];
        }
        uint32_t x = loc;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const uint32_t y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        uint32_t pre = x - loc;
#pragma unroll
        for (int e = 0; e < 3; ++e) {
            const int q = 3 * lane + e;
            if (q < NRV) above[NRV - 1 - q] = (uint16_t)pre;
            pre += h[e];
        }
    }
    __syncthreads();
    uint32_t tile_sum = 0;
#pragma unroll
    for (int k = 0; k < AK_PER; ++k) {
        const int64_t t = t0 + 64 * k + lane;
        if (t >= N) continue;
        const unsigned long long* mm = m[r[k]];
        uint32_t pos = above[r[k]] + __popcll(mm[k] & ((1ull << lane) - 1ull));
#pragma unroll
        for (int j = 0; j < AK_PER - 1; ++j)
            if (j < k) pos += __popcll(mm[j]);
        srank[t0 + pos] = (uint8_t)r[k];
        sidx[t0 + pos] = (uint32_t)t;
        // the chunk's storage: each tile of 16 positions takes 16 x its first (largest) rank
        if ((pos & 15) == 0) tile_sum += 16u * r[k];
    }
    return wave_sum(tile_sum);
}

// ---- 6. threshold, final ranks, each chunk's size ------------------------------------------------
// Per-head codec (ORDER): 8-bit ranks, each chunk's storage order (srank, sidx) and its size in
// tile rectangles.  Shared basis: 16-bit ranks in original order and each chunk's rank sum.
// The chunk sizes go to csum[c] (unscanned: the scan runs in whichever pass reads them next).
template <typename RT, bool ORDER>
__global__ __launch_bounds__(AK_T) void al_final(int64_t N, const uint32_t* __restrict__ u_ws,
                                                 const uint64_t* __restrict__ phi_ws,
                                                 const uint64_t* __restrict__ cand, RT* __restrict__ rank,
                                                 uint8_t* __restrict__ srank, uint32_t* __restrict__ sidx,
                                                 uint32_t* __restrict__ csum, const AlCtl* __restrict__ ctl) {
    __shared__ AlSelSmem ss;
    // storage order of each wave's chunk: per-rank 256-bit token masks, and the count of
    // tokens of higher rank per rank value
    __shared__ unsigned long long msk[ORDER ? AK_T / 64 : 1][NRV][4];
    __shared__ uint16_t above_r[ORDER ? AK_T / 64 : 1][NRV];
    // every load of the pass goes out first: the tokens, one list entry per thread
    const int64_t ti = (int64_t)threadIdx.x < N ? (int64_t)threadIdx.x : N - 1;
    const uint64_t my_hi = cand[2 * ti], my_lo = cand[2 * ti + 1];
    uint64_t phi[AK_PER];
    uint32_t u[AK_PER], r[AK_PER];
#pragma unroll
    for (int k = 0; k < AK_PER; ++k) {
        const int64_t t = al_tok(k), tt = t < N ? t : N - 1;
        phi[k] = phi_ws[tt];
        u[k] = u_ws[tt];
        r[k] = rank[tt];
    }
    uint64_t T_hi, T_lo;
    al_threshold(N, cand, ctl, my_hi, my_lo, ss, T_hi, T_lo);
    const bool any = ctl->any;
#pragma unroll
    for (int k = 0; k < AK_PER; ++k) {
        const int64_t t = al_tok(k);
        if (t >= N) continue;
        if (any && phi[k] != CAPPED) {
            const bool take = phi[k] > T_hi || (phi[k] == T_hi && lo_key(u[k], t) >= T_lo);
            if (take) {
                r[k] += 1;
                rank[t] = (RT)r[k];
            }
        }
    }
    const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int64_t c = (int64_t)blockIdx.x * (AK_TOK / CHUNK) + wv;
    uint32_t size;
    if constexpr (ORDER) {
        size = chunk_order(msk[wv], above_r[wv], r, c * CHUNK, N, srank, sidx);
    } else {
        uint32_t sum = 0;
#pragma unroll
        for (int k = 0; k < AK_PER; ++k)
            if (al_tok(k) < N) sum += r[k];
        size = wave_sum(sum);
    }
    if (lane == 0 && c * CHUNK < N) csum[c] = size;
}

// Exclusive prefix of the chunk sizes up to chunk c (c + 1 <= n_chunks) by one wave.
// Eight independent loads per lane at a time (clamped addresses, masked values).
__device__ __forceinline__ uint32_t chunk_prefix(const uint32_t* __restrict__ csum, int64_t c) {
    const int lane = threadIdx.x & 63;
    uint32_t pre = 0;
    for (int64_t i0 = 0; i0 < c; i0 += 8 * 64) {
        uint32_t v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int64_t i = i0 + 64 * j + lane;
            v[j] = csum[i < c ? i : 0];
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) pre += i0 + 64 * j + lane < c ? v[j] : 0u;
    }
    return wave_sum(pre);
}

// ---- 7. shared basis: chunk offsets and per-token offsets = chunk offset + the chunk's
//         earlier ranks (one wave per chunk, which scans the chunk sums before it itself)
__global__ __launch_bounds__(AK_T) void al_offsets(int64_t N, const uint16_t* __restrict__ rank,
                                                   const uint32_t* __restrict__ csum,
                                                   uint32_t* __restrict__ chunk_off,
                                                   uint32_t* __restrict__ offset, int n_chunks) {
    const int lane = threadIdx.x & 63;
    const int64_t c = (int64_t)blockIdx.x * (AK_TOK / CHUNK) + (threadIdx.x >> 6);
    if (c * CHUNK >= N) return;
    uint32_t pre = chunk_prefix(csum, c);
    if (lane == 0) chunk_off[c] = pre;
#pragma unroll
    for (int k = 0; k < AK_PER; ++k) {
        const int64_t t = c * CHUNK + 64 * k + lane;       // the wave's tokens, in index order
        const uint32_t r = t < N ? rank[t] : 0u;
        uint32_t x = r;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const uint32_t y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        if (t < N) offset[t] = pre + x - r;
        pre += __shfl(x, 63, 64);
    }
    if (c == n_chunks - 1 && lane == 0) {       // the totals
        chunk_off[n_chunks] = pre;
        offset[N] = pre;
    }
}

// ---- 7'. chunk offsets for the allocation entry point (chunk sizes -> exclusive prefix,
//          total at [n_chunks]); the compress path leaves this scan to the projection
constexpr int SCAN_T = 1024;
constexpr int SCAN_PT = MAX_CODED_CHUNKS / SCAN_T;   // chunk sums per thread

__global__ __launch_bounds__(SCAN_T) void al_scan(const uint32_t* __restrict__ csum,
                                                  uint32_t* __restrict__ chunk_off, int n_chunks) {
    __shared__ uint32_t wt32[SCAN_T / 64];
    const int per = (n_chunks + SCAN_T - 1) / SCAN_T;
    const int i0 = per * threadIdx.x;
    uint32_t v[SCAN_PT], loc = 0;
#pragma unroll
    for (int j = 0; j < SCAN_PT; ++j) {
        v[j] = j < per && i0 + j < n_chunks ? csum[i0 + j] : 0u;
        loc += v[j];
    }
    uint32_t total;
    uint32_t pre = block_exscan<SCAN_T, uint32_t>(loc, wt32, total);
#pragma unroll
    for (int j = 0; j < SCAN_PT; ++j)
        if (j < per && i0 + j < n_chunks) {
            chunk_off[i0 + j] = pre;
            pre += v[j];
        }
    if (threadIdx.x == 0) chunk_off[n_chunks] = total;
}

hipError_t launch_allocate(const varrate_shape& sh, const float* sbar, varrate_cache& c,
                           uint8_t* ws, hipStream_t st, const float* s_part, const uint32_t** chunk_sizes) {
    const int64_t N = sh.n - sh.w;
    const int R = D, r_min = sh.r_min;
    const int64_t B = c.B;
    const int nwg = (int)((N + AK_TOK - 1) / AK_TOK);
    const int n_chunks = (int)((N + CHUNK - 1) / CHUNK);
    if (n_chunks > MAX_CODED_CHUNKS) return hipErrorInvalidValue;
    const AlWs w = al_ws(ws, N);
    if (s_part)
        al_pool_minmax<<<nwg, AK_T, 0, st>>>(s_part, N, sh.G, salience_pool_scale(sh), const_cast<float*>(sbar),
                                             w.mm, w.clear, w.clear_words);
    else
        al_minmax<<<nwg, AK_T, 0, st>>>(sbar, N, w.mm, w.clear, w.clear_words);
    al_weights<<<nwg, AW_T, 0, st>>>(sbar, N, w.mm, nwg, w.u, w.c_pack, w.ctl);
    al_fine<<<nwg, AW_T, 0, st>>>(N, B, r_min, R, w.u, w.c_pack, w.f_cnt, w.ctl);
    al_floors<uint8_t><<<nwg, AW_T, 0, st>>>(N, B, r_min, R, w.u, w.f_cnt, c.rank, w.phi, w.d_cnt, w.ctl);
    al_gather<<<nwg, AK_T, 0, st>>>(N, B, w.u, w.phi, w.d_cnt, w.cand, w.ctl);
    al_final<uint8_t, true><<<nwg, AK_T, 0, st>>>(N, w.u, w.phi, w.cand, c.rank, c.srank, c.sidx, w.csum, w.ctl);
    if (chunk_sizes)
        *chunk_sizes = w.csum;
    else
        al_scan<<<1, SCAN_T, 0, st>>>(w.csum, c.chunk_off, n_chunks);
    return hipGetLastError();
}

hipError_t launch_allocate_joint(const varrate_shape& sh, int R, int64_t B, const float* sbar, uint16_t* rank,
                                 uint32_t* offset, uint32_t* chunk_off, uint8_t* ws, hipStream_t st,
                                 const float* s_part) {
    const int64_t N = sh.n - sh.w;
    const int r_min = sh.r_min;
    const int nwg = (int)((N + AK_TOK - 1) / AK_TOK);
    const int n_chunks = (int)((N + CHUNK - 1) / CHUNK);
    if (n_chunks > MAX_CODED_CHUNKS) return hipErrorInvalidValue;
    const AlWs w = al_ws(ws, N);
    if (s_part)
        al_pool_minmax<<<nwg, AK_T, 0, st>>>(s_part, N, sh.G, salience_pool_scale(sh), const_cast<float*>(sbar),
                                             w.mm, w.clear, w.clear_words);
    else
        al_minmax<<<nwg, AK_T, 0, st>>>(sbar, N, w.mm, w.clear, w.clear_words);
    al_weights<<<nwg, AW_T, 0, st>>>(sbar, N, w.mm, nwg, w.u, w.c_pack, w.ctl);
    al_fine<<<nwg, AW_T, 0, st>>>(N, B, r_min, R, w.u, w.c_pack, w.f_cnt, w.ctl);
    al_floors<uint16_t><<<nwg, AW_T, 0, st>>>(N, B, r_min, R, w.u, w.f_cnt, rank, w.phi, w.d_cnt, w.ctl);
    al_gather<<<nwg, AK_T, 0, st>>>(N, B, w.u, w.phi, w.d_cnt, w.cand, w.ctl);
    al_final<uint16_t, false><<<nwg, AK_T, 0, st>>>(N, w.u, w.phi, w.cand, rank, nullptr, nullptr, w.csum, w.ctl);
    al_offsets<<<nwg, AK_T, 0, st>>>(N, rank, w.csum, chunk_off, offset, n_chunks);
    return hipGetLastError();
}

}  // namespace vr
