// Rank-space decode attention over the compressed cache, gfx950.
//
// Attention over the reconstructed cache of Eq. (6) without reconstructing it: with an
// orthonormal key basis <q, P_K^T (m . c)> = <P_K q, m . c>, and the value side is linear,
// so  o = P_V^T (sum_t p_t m_t . c^V_t) + sum_e p_e v_e.
//
// Grid (n_wg + 1, G * nqt, S).  Workgroup x = 0 attends to the exact slots (window +
// appended tokens) in the original space; workgroup x >= 1 streams the 16-token tiles
// [(x-1) tpw, x tpw) of KV head g's stored tokens (tile t = chunk t/16, slots 16 (t%16)..),
// for one sequence and one tile of up to 16 query rows (row = query * H/G + head).  Per workgroup (8 waves, two workgroups per CU):
//   1. q' = P_K[g] q / sqrt(d) by MFMA (basis split into bf16 hi + lo parts, ~2^-16 error),
//      while the chunks' stored ranks are fetched with one vector load per 16 tokens;
//   2. waves take 16-token tiles of the rank-sorted storage.  Each lane gathers its MFMA
//      operands straight from the packed ragged rows: 16-byte row segments for the score
//      tile (16 tokens x 32 coefficients per step, masked past each token's rank) and, for
//      the value tile, 4 tokens' coefficients at one rank index.  The score C fragment
//      (lane = query row, 4 tokens) is exactly the A fragment of the 16x16x16 value MFMA,
//      so the online softmax needs no shuffles; p is split into bf16 hi + lo parts;
//   3. the waves' (max, sum, acc) are combined in a fixed order into one partial record;
//   4. a second launch (one workgroup per sequence, head and row tile) loads every partial
//      with coalesced vector loads, merges them by log-sum-exp, rotates the rank-space sum
//      back with P_V^T (MFMA) and adds the exact part.
// A tile's first token has the largest rank (storage is rank-descending per chunk), which
// bounds its MFMA steps: ceil(r_max/32) score steps and ceil(r_max/16) value blocks.
#include "vr_internal.h"

namespace vr {

constexpr int DC_THREADS = 512;
constexpr int DC_WAVES = 8;
constexpr int DC_SEQ = 16;                 // sequences per launch (descriptors in kernargs)
constexpr int DC_REC = 16 + 16 + 16 * D;   // floats per partial record: m, l, acc[16][128]
constexpr int DC_MAX_CPW = 16;            // chunks one workgroup's tile range may touch
constexpr int DC_MAX_REC = 512;            // partial records per (sequence, head, row tile)

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f32x4 mfma16(u32x2 a, u32x2 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, a),
                                                     __builtin_bit_cast(s16x4, b), c, 0, 0, 0);
}

struct DecSeq {
    const void* coef_k;
    const void* coef_v;
    const uint8_t* srank;
    const uint32_t* chunk_off;
    const void* k_exact;
    const void* v_exact;
    const void* q;
    void* out;
    int64_t n_exact;
};

struct DecParams {
    DecSeq seq[DC_SEQ];
    const float* PK;
    const float* PV;
    float* part;
    int64_t N, coef_stride, cap;
    int G, H, hpg, nqt, rows_total, n_chunks, cpw, n_wg, tpw, total_tiles;
};

template <bool F32> struct Elem;
template <> struct Elem<false> { typedef uint16_t T; };
template <> struct Elem<true> { typedef float T; };

// 8 consecutive elements at p (nv of them valid) as bf16 (hi, lo) fragments.
template <bool F32>
__device__ __forceinline__ void load_row8(const typename Elem<F32>::T* p, int nv, u32x4& hi, u32x4& lo) {
    if constexpr (!F32) {
        hi = nv > 0 ? keep_first(load16_a2(p), nv) : u32x4{0, 0, 0, 0};
        lo = u32x4{0, 0, 0, 0};
    } else {
        float x[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        if (nv > 0) {
            u32x4 a, b;
            __builtin_memcpy(&a, p, 16);
            __builtin_memcpy(&b, p + 4, 16);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                x[e] = e < nv ? __uint_as_float(a[e]) : 0.f;
                x[4 + e] = 4 + e < nv ? __uint_as_float(b[e]) : 0.f;
            }
        }
        split8(x, hi, lo);
    }
}

// 4 fp32 -> bf16x4 (hi, lo)
__device__ __forceinline__ void split4(const float* x, u32x2& hi, u32x2& lo) {
    uint32_t h[4], l[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) split_bf16(x[e], h[e], l[e]);
    hi = u32x2{pack2(h[0], h[1]), pack2(h[2], h[3])};
    lo = u32x2{pack2(l[0], l[1]), pack2(l[2], l[3])};
}

struct DecSmem {
    float* qp;        // [16][128] query rows (rotated or scaled); merge: partial lanes
    u32x4* qf;        // [4 steps][hi, lo][64 lanes] score B-operand fragments
    float* comb;      // [4][nr4][128]; merge: accR [nr4][128], accE [nr4][128]
    float* cm;        // [8][16]
    float* cl;        // [8][16]
    float* mrow;      // [16]
    float* lrow;      // [16]
    uint32_t* cb;     // [DC_MAX_CPW]
    int* cT;          // [DC_MAX_CPW]
    int* flag;        // [4]
    uint8_t* sr;      // [cpw][256]
    uint16_t* so;     // [cpw][256]
};

__device__ __forceinline__ DecSmem carve(uint8_t* smem, int nr4, int cpw) {
    DecSmem s;
    float* f = reinterpret_cast<float*>(smem);
    s.qp = f; f += 16 * D;
    s.qf = reinterpret_cast<u32x4*>(f); f += 4 * 2 * 64 * 4;
    s.comb = f; f += 4 * nr4 * D;
    s.cm = f; f += DC_WAVES * 16;
    s.cl = f; f += DC_WAVES * 16;
    s.mrow = f; f += 16;
    s.lrow = f; f += 16;
    uint32_t* u = reinterpret_cast<uint32_t*>(f);
    s.cb = u; u += DC_MAX_CPW;
    s.cT = reinterpret_cast<int*>(u); u += DC_MAX_CPW;
    u += DC_MAX_CPW + 4;
    s.flag = reinterpret_cast<int*>(u); u += 4;
    s.sr = reinterpret_cast<uint8_t*>(u);                 // 16-byte aligned (sizes above)
    s.so = reinterpret_cast<uint16_t*>(s.sr + cpw * CHUNK);
    return s;
}

static inline size_t decode_smem_bytes(int nr4, int cpw) {
    return (size_t)(16 * D + 4 * 2 * 64 * 4 + 4 * nr4 * D + 2 * DC_WAVES * 16 + 32) * 4 +
           (size_t)(3 * DC_MAX_CPW + 8) * 4 + (size_t)cpw * CHUNK * 3;
}

template <bool F32>
__global__ __launch_bounds__(DC_THREADS, F32 ? 2 : 4) void decode_kernel(DecParams p) {
    typedef typename Elem<F32>::T ET;
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    const int x = blockIdx.x, gq = blockIdx.y, sq = blockIdx.z;
    const int g = gq / p.nqt, qt = gq % p.nqt;
    const DecSeq& S = p.seq[sq];
    const int rows = min(16, p.rows_total - 16 * qt);
    const int nr4 = (rows + 3) & ~3;
    const bool exact = x == 0;          // dispatched first; the coded groups follow
    const int xc = x - 1;               // coded chunk group
    const int cpw = p.cpw;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int grp = lane >> 4, col = lane & 15;
    DecSmem sm = carve(smem, nr4, cpw);
    const float scale = 0.08838834764831845f;  // 1/sqrt(128)
    const ET* qsrc = reinterpret_cast<const ET*>(S.q);

    // ---- 1a. issue the basis rows and query rows the rotation needs
    const float* P = p.PK + (int64_t)g * D * D;
    const int qrow_l = 16 * qt + col;
    const bool q_ok = qrow_l < p.rows_total;
    const int query_l = q_ok ? qrow_l / p.hpg : 0, hh_l = q_ok ? qrow_l % p.hpg : 0;
    const ET* qv = qsrc + ((int64_t)query_l * p.H + g * p.hpg + hh_l) * D;
    u32x4 pa[4][2];
    u32x4 qb[4][2];
    if (!exact) {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const float* src = P + (16 * wave + col) * D + 32 * s + 8 * grp;
            pa[s][0] = load16(src);
            pa[s][1] = load16(src + 4);
            load_row8<F32>(qv + 32 * s + 8 * grp, q_ok ? 8 : 0, qb[s][0], qb[s][1]);
        }
    }
    // ---- 1b. stored ranks and chunk bases of the chunks this tile range touches
    const int tau0 = exact ? 0 : xc * p.tpw;
    const int tau1 = exact ? 0 : min(tau0 + p.tpw, p.total_tiles);
    const int c_lo = tau0 >> 4;
    const int ncl = exact ? 0 : ((tau1 - 1) >> 4) - c_lo + 1;
    if (!exact) {
        const int64_t t_beg = (int64_t)c_lo * CHUNK;
        for (int idx = tid; idx < ncl * (CHUNK / 16); idx += DC_THREADS) {
            const int64_t t = t_beg + (int64_t)idx * 16;
            u32x4 v = {0, 0, 0, 0};
            if (t < p.N) v = load16(S.srank + t);      // srank is padded to a multiple of 64
            *reinterpret_cast<u32x4*>(sm.sr + idx * 16) = v;
        }
        if (tid < ncl) {
            const int c = c_lo + tid;
            const int64_t t0 = (int64_t)c * CHUNK;
            sm.cT[tid] = (int)((p.N - t0) < CHUNK ? (p.N - t0) : CHUNK);
            sm.cb[tid] = S.chunk_off[c];
        }
    }
    // ---- 1c. query rows: rotated into the key basis (coded) or as is (exact)
    if (!exact) {
        f32x4 c = {0, 0, 0, 0};
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            float a8[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) { a8[e] = __uint_as_float(pa[s][0][e]); a8[4 + e] = __uint_as_float(pa[s][1][e]); }
            u32x4 ah, al;
            split8(a8, ah, al);
            c = mfma(ah, qb[s][0], c);
            c = mfma(al, qb[s][0], c);
            if constexpr (F32) c = mfma(ah, qb[s][1], c);
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) sm.qp[col * D + 16 * wave + 4 * grp + v] = c[v] * scale;
    } else {
        for (int idx = tid; idx < 16 * D; idx += DC_THREADS) {
            const int r = idx / D, i = idx % D;
            const int qrow = 16 * qt + r;
            float val = 0.f;
            if (qrow < p.rows_total) {
                const int query = qrow / p.hpg, hh = qrow % p.hpg;
                const ET e = qsrc[((int64_t)query * p.H + g * p.hpg + hh) * D + i];
                if constexpr (F32) val = e; else val = bf16_to_f32(e);
            }
            sm.qp[idx] = val * scale;
        }
    }
    __syncthreads();
    // ---- 1d. local offsets (exclusive scan of the stored ranks inside each chunk)
    for (int cc = wave; cc < ncl; cc += DC_WAVES) {
        uint32_t r[4], loc = 0;
        const int T = sm.cT[cc];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            r[e] = 4 * lane + e < T ? sm.sr[cc * CHUNK + 4 * lane + e] : 0;
            loc += r[e];
        }
        uint32_t xs = loc;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            uint32_t y = __shfl_up(xs, off, 64);
            if (lane >= off) xs += y;
        }
        uint32_t pre = xs - loc;
#pragma unroll
        for (int e = 0; e < 4; ++e) { sm.so[cc * CHUNK + 4 * lane + e] = (uint16_t)pre; pre += r[e]; }
    }
    // ---- 2. score-operand fragments (shared by all waves): lane -> query row col, K group grp
    {
        const int s = tid >> 7, part = (tid >> 6) & 1;   // 512 threads <-> 4 steps x {hi, lo} x 64 lanes
        float v8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v8[e] = sm.qp[col * D + 32 * s + 8 * grp + e];
        u32x4 h, l;
        split8(v8, h, l);
        sm.qf[(s * 2 + part) * 64 + lane] = part ? l : h;
    }
    __syncthreads();

    const int t_first = exact ? 0 : tau0;
    const int t_end = exact ? (int)((S.n_exact + 15) / 16) : tau1;
    const ET* kbase_all = reinterpret_cast<const ET*>(exact ? S.k_exact : S.coef_k);
    const ET* vbase_all = reinterpret_cast<const ET*>(exact ? S.v_exact : S.coef_v);
    float m_run = -INFINITY, l_part = 0.f;
    f32x4 acc[8];
#pragma unroll
    for (int b = 0; b < 8; ++b) acc[b] = f32x4{0, 0, 0, 0};

    for (int tile = t_first + wave; tile < t_end; tile += DC_WAVES) {
        int cc = 0, i0, T, rmax;
        int64_t base;
        if (exact) {
            i0 = tile * 16;
            T = (int)S.n_exact;
            rmax = D;
            base = (int64_t)g * p.cap * D;
        } else {
            cc = (tile >> 4) - c_lo;
            i0 = (tile & 15) * 16;
            T = sm.cT[cc];
            rmax = sm.sr[cc * CHUNK + i0];
            base = (int64_t)g * p.coef_stride + sm.cb[cc];
        }
        const ET* Kb = kbase_all + base;
        const ET* Vb = vbase_all + base;
        const int ks = (rmax + 31) >> 5, nb = (rmax + 15) >> 4;
        // token metadata: rank and offset of stored slot i (0 rank past the chunk's end)
        auto meta = [&](int i, int& r, int& o) {
            if (i >= T) { r = 0; o = 0; return; }
            if (exact) { r = D; o = i * D; }
            else { r = sm.sr[cc * CHUNK + i]; o = sm.so[cc * CHUNK + i]; }
        };
        // score operand: row = token i0 + col, coefficients 32 s + 8 grp .. + 7
        int rk, ok_;
        meta(i0 + col, rk, ok_);
        u32x4 kh[4], kl[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            if (s < ks) {
                const int c0 = 32 * s + 8 * grp;
                int nv = rk - c0;
                nv = nv < 0 ? 0 : (nv > 8 ? 8 : nv);
                load_row8<F32>(Kb + ok_ + c0, nv, kh[s], kl[s]);
            } else {
                kh[s] = kl[s] = u32x4{0, 0, 0, 0};
            }
        }
        // value operand: column j = 16 b + col, tokens i0 + 4 grp + e
        int vr_[4], vo_[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) meta(i0 + 4 * grp + e, vr_[e], vo_[e]);
        u32x2 vh[8], vl[8];
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            if (b < nb) {
                const int j = 16 * b + col;
                if constexpr (F32) {
                    float f4[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) f4[e] = j < vr_[e] ? Vb[vo_[e] + j] : 0.f;
                    split4(f4, vh[b], vl[b]);
                } else {
                    uint32_t h[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) h[e] = j < vr_[e] ? (uint32_t)Vb[vo_[e] + j] : 0u;
                    vh[b] = u32x2{pack2(h[0], h[1]), pack2(h[2], h[3])};
                    vl[b] = u32x2{0, 0};
                }
            } else {
                vh[b] = vl[b] = u32x2{0, 0};
            }
        }
        // scores: C lane -> query row col, tokens i0 + 4 grp + v
        f32x4 sc = {0, 0, 0, 0};
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            if (s < ks) {
                const u32x4 qh = sm.qf[(s * 2) * 64 + lane], ql = sm.qf[(s * 2 + 1) * 64 + lane];
                sc = mfma(kh[s], qh, sc);
                sc = mfma(kh[s], ql, sc);
                if constexpr (F32) sc = mfma(kl[s], qh, sc);
            }
        }
        float sv[4];
        float tmax = -INFINITY;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            sv[v] = i0 + 4 * grp + v < T ? sc[v] : -INFINITY;
            tmax = fmaxf(tmax, sv[v]);
        }
        tmax = fmaxf(tmax, shfl_xor_f(tmax, 16));
        tmax = fmaxf(tmax, shfl_xor_f(tmax, 32));
        const float m_new = fmaxf(m_run, tmax);
        if (__ballot(m_new > m_run)) {
            const float alpha = m_new > m_run ? fast_exp(m_run - m_new) : 1.f;
            l_part *= alpha;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const float av = __shfl(alpha, 4 * grp + v, 64);
#pragma unroll
                for (int b = 0; b < 8; ++b) acc[b][v] *= av;
            }
            m_run = m_new;
        }
        float pv[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            pv[v] = m_run == -INFINITY ? 0.f : fast_exp(sv[v] - m_run);
            l_part += pv[v];
        }
        u32x2 ph, pl;
        split4(pv, ph, pl);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            if (b < nb) {
                acc[b] = mfma16(ph, vh[b], acc[b]);
                acc[b] = mfma16(pl, vh[b], acc[b]);
                if constexpr (F32) acc[b] = mfma16(ph, vl[b], acc[b]);
            }
        }
    }

    // ---- 3. combine the waves of this workgroup (fixed order)
    float lsum = l_part + shfl_xor_f(l_part, 16);
    lsum += shfl_xor_f(lsum, 32);
    if (lane < 16) { sm.cm[wave * 16 + col] = m_run; sm.cl[wave * 16 + col] = lsum; }
    __syncthreads();
    if (tid < 16) {
        float M = -INFINITY;
        for (int w = 0; w < DC_WAVES; ++w) M = fmaxf(M, sm.cm[w * 16 + tid]);
        float L = 0.f;
        for (int w = 0; w < DC_WAVES; ++w) {
            const float mw = sm.cm[w * 16 + tid];
            L += mw == -INFINITY ? 0.f : sm.cl[w * 16 + tid] * fast_exp(mw - M);
        }
        sm.mrow[tid] = M;
        sm.lrow[tid] = L;
    }
    __syncthreads();
    float fac[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const int row = 4 * grp + v;
        const float mw = sm.cm[wave * 16 + row];
        fac[v] = mw == -INFINITY ? 0.f : fast_exp(mw - sm.mrow[row]);
    }
    if (wave >= 4) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int row = 4 * grp + v;
            if (row < nr4) {
#pragma unroll
                for (int b = 0; b < 8; ++b) sm.comb[((wave - 4) * nr4 + row) * D + 16 * b + col] = acc[b][v] * fac[v];
            }
        }
    }
    __syncthreads();
    if (wave < 4) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int row = 4 * grp + v;
            if (row < nr4) {
#pragma unroll
                for (int b = 0; b < 8; ++b) {
                    float* dst = &sm.comb[(wave * nr4 + row) * D + 16 * b + col];
                    *dst = acc[b][v] * fac[v] + *dst;
                }
            }
        }
    }
    __syncthreads();
    const int units = p.G * p.nqt;
    const int nrec = p.n_wg + 1;
    float* recs = p.part + ((int64_t)sq * units + gq) * nrec * DC_REC;
    {
        float* rec = recs + (int64_t)x * DC_REC;
        const int n4 = nr4 * D / 4;
        for (int idx = tid; idx < n4; idx += DC_THREADS) {
            const f32x4 a = reinterpret_cast<const f32x4*>(sm.comb)[idx];
            const f32x4 b = reinterpret_cast<const f32x4*>(sm.comb + nr4 * D)[idx];
            const f32x4 c = reinterpret_cast<const f32x4*>(sm.comb + 2 * nr4 * D)[idx];
            const f32x4 d = reinterpret_cast<const f32x4*>(sm.comb + 3 * nr4 * D)[idx];
            reinterpret_cast<f32x4*>(rec + 32)[idx] = ((a + b) + c) + d;
        }
        if (tid < 16) { rec[tid] = sm.mrow[tid]; rec[16 + tid] = sm.lrow[tid]; }
    }

}


// ----------------------------------------------------------------------------------------
// Merge of the partial records of one (sequence, KV head, row tile): log-sum-exp over the
// records (record 0 = exact slots, original space; records 1.. = coded chunk groups, rank
// space), back-rotation of the rank-space sum with P_V^T by MFMA, division by the softmax
// denominator.  A separate launch: the kernel boundary publishes every record, so no
// workgroup of the streaming kernel needs a device-wide fence.
struct MergeParams {
    const float* part;
    const float* PV;
    void* out;              // [S][Q][H][d] of this launch's sequences
    int64_t out_seq_stride; // elements per sequence
    int G, H, hpg, nqt, rows_total, n_wg;
};

template <bool F32>
__global__ __launch_bounds__(DC_THREADS) void decode_merge_kernel(MergeParams p) {
    typedef typename Elem<F32>::T ET;
    __shared__ float wm[DC_MAX_REC * 16];
    __shared__ float wl[DC_MAX_REC * 16];
    __shared__ __attribute__((aligned(16))) float lanes[DC_THREADS * 4];
    __shared__ __attribute__((aligned(16))) float accR[16 * D];
    __shared__ __attribute__((aligned(16))) float accE[16 * D];
    __shared__ float mrow[16], lrow[16];
    const int unit = blockIdx.x;
    const int units = p.G * p.nqt;
    const int sq = unit / units, gq = unit % units;
    const int g = gq / p.nqt, qt = gq % p.nqt;
    const int rows = min(16, p.rows_total - 16 * qt);
    const int nr4 = (rows + 3) & ~3;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int grp = lane >> 4, col = lane & 15;
    const int nrec = p.n_wg + 1;
    const float* recs = p.part + (int64_t)unit * nrec * DC_REC;

    // per-record maxima and sums
    for (int idx = tid; idx < nrec * 16; idx += DC_THREADS) {
        const int r = idx >> 4, row = idx & 15;
        wm[idx] = recs[(int64_t)r * DC_REC + row];
        wl[idx] = recs[(int64_t)r * DC_REC + 16 + row];
    }
    __syncthreads();
    if (tid < 16) {
        float M = -INFINITY;
        for (int r = 0; r < nrec; ++r) M = fmaxf(M, wm[r * 16 + tid]);
        mrow[tid] = M;
    }
    __syncthreads();
    for (int idx = tid; idx < nrec * 16; idx += DC_THREADS) {
        const float m = wm[idx];
        wm[idx] = m == -INFINITY ? 0.f : fast_exp(m - mrow[idx & 15]);
    }
    __syncthreads();
    if (tid < 16) {
        float L = 0.f;
        for (int r = 0; r < nrec; ++r) L += wm[r * 16 + tid] * wl[r * 16 + tid];
        lrow[tid] = L;
    }
    // weighted sum of the coded records: thread -> (float4 e, record lane k)
    const int E = nr4 * D / 4;                  // float4s per record
    const int KL = DC_THREADS / E;              // record lanes
    {
        const int e = tid % E, k = tid / E;
        const int row = (e * 4) / D;
        f32x4 s4 = {0, 0, 0, 0};
        if (k < KL) {
            for (int r0 = 1 + k; r0 < nrec; r0 += 8 * KL) {
                f32x4 a[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) {      // eight independent loads in flight
                    const int r = r0 + u * KL;
                    a[u] = r < nrec ? reinterpret_cast<const f32x4*>(recs + (int64_t)r * DC_REC + 32)[e]
                                    : f32x4{0, 0, 0, 0};
                }
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int r = r0 + u * KL;
                    s4 += (r < nrec ? wm[r * 16 + row] : 0.f) * a[u];
                }
            }
        }
        reinterpret_cast<f32x4*>(lanes)[tid] = s4;
    }
    __syncthreads();
    if (tid < E) {
        f32x4 t = reinterpret_cast<const f32x4*>(lanes)[tid];
        for (int kk = 1; kk < KL; ++kk) t += reinterpret_cast<const f32x4*>(lanes)[kk * E + tid];
        reinterpret_cast<f32x4*>(accR)[tid] = t;
        const f32x4 ex = reinterpret_cast<const f32x4*>(recs + 32)[tid];
        reinterpret_cast<f32x4*>(accE)[tid] = wm[(tid * 4) / D] * ex;
    }
    __syncthreads();
    // back-rotation by MFMA: C[row][c] = sum_j accR[row][j] P_V[j][c]
    // wave -> column block 16 wave.., lane -> column col, K group grp
    const float* PV = p.PV + (int64_t)g * D * D;
    float pb[4][8];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < 8; ++i) pb[s][i] = PV[(32 * s + 8 * grp + i) * D + 16 * wave + col];
    f32x4 o = {0, 0, 0, 0};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        float a8[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) a8[i] = col < nr4 ? accR[col * D + 32 * s + 8 * grp + i] : 0.f;
        u32x4 ah, al, bh, bl;
        split8(a8, ah, al);
        split8(pb[s], bh, bl);
        o = mfma(ah, bh, o);
        o = mfma(al, bh, o);
        o = mfma(ah, bl, o);
    }
    // C lane -> column c = 16 wave + col, rows 4 grp + v
    ET* out = reinterpret_cast<ET*>(p.out) + (int64_t)sq * p.out_seq_stride;
    const int c = 16 * wave + col;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const int row = 4 * grp + v;
        if (row < rows) {
            const float val = (o[v] + accE[row * D + c]) / lrow[row];
            const int qrow = 16 * qt + row;
            const int query = qrow / p.hpg, hh = qrow % p.hpg;
            const int64_t oi = ((int64_t)query * p.H + g * p.hpg + hh) * D + c;
            if constexpr (F32) out[oi] = val;
            else out[oi] = (uint16_t)f32_to_bf16(val);
        }
    }
}
// ----------------------------------------------------------------------------------------
struct DecPlan {
    int nqt, n_chunks, cpw, n_wg, tpw, total_tiles;
};

static DecPlan plan_decode(const varrate_shape& sh, int S, int Q) {
    DecPlan pl;
    const int64_t N = sh.n - sh.w;
    const int rows_total = Q * (sh.H / sh.G);
    pl.nqt = (rows_total + 15) / 16;
    pl.n_chunks = (int)((N + CHUNK - 1) / CHUNK);
    const int64_t last = N - (int64_t)(pl.n_chunks - 1) * CHUNK;
    pl.total_tiles = 16 * (pl.n_chunks - 1) + (int)((last + 15) / 16);
    const int units = (S < DC_SEQ ? S : DC_SEQ) * sh.G * pl.nqt;
    // coded workgroups + one exact workgroup per unit: about two workgroups per CU, at
    // least one tile per wave, at most (DC_MAX_CPW - 1) chunks of tiles per workgroup
    int n_wg = 512 / (units > 0 ? units : 1) - 1;
    const int by_waves = (pl.total_tiles + DC_WAVES - 1) / DC_WAVES;
    const int max_tpw = (DC_MAX_CPW - 1) * 16;
    const int by_span = (pl.total_tiles + max_tpw - 1) / max_tpw;
    n_wg = n_wg > by_waves ? by_waves : n_wg;
    n_wg = n_wg < by_span ? by_span : n_wg;
    n_wg = n_wg < 1 ? 1 : n_wg;
    pl.tpw = (pl.total_tiles + n_wg - 1) / n_wg;
    pl.n_wg = (pl.total_tiles + pl.tpw - 1) / pl.tpw;
    pl.cpw = (pl.tpw + 15) / 16 + 1;    // chunks a tile range can touch
    return pl;
}

// Workspace: the partial records of every (sequence, KV head, row tile).
size_t decode_units(const varrate_shape& sh, int S, int Q) {
    return (size_t)S * sh.G * plan_decode(sh, S, Q).nqt;
}

bool decode_supported(const varrate_shape& sh, int S, int Q) {
    return plan_decode(sh, S, Q).n_wg + 1 <= DC_MAX_REC;
}

size_t decode_ws_bytes(const varrate_shape& sh, int S, int Q) {
    DecPlan pl = plan_decode(sh, S, Q);
    const size_t units = (size_t)S * sh.G * pl.nqt;
    return align256(units * (pl.n_wg + 1) * DC_REC * sizeof(float));
}

template <bool F32>
static hipError_t set_smem_attr(size_t bytes) {
    static size_t done = 0;
    if (bytes <= done) return hipSuccess;
    hipError_t e = hipFuncSetAttribute((const void*)decode_kernel<F32>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e == hipSuccess) done = bytes;
    return e;
}

hipError_t launch_decode(const varrate_shape& sh, const varrate_cache* caches, int S, const void* q,
                         int Q, const float* PK, const float* PV, void* out, uint8_t* ws,
                         hipStream_t st) {
    DecPlan pl = plan_decode(sh, S, Q);
    const int hpg = sh.H / sh.G;
    const int rows_total = Q * hpg;
    const size_t units_all = (size_t)S * sh.G * pl.nqt;
    if (pl.n_wg + 1 > DC_MAX_REC) return hipErrorInvalidValue;
    (void)units_all;
    float* part = (float*)ws;
    const size_t es = sh.dtype == VARRATE_BF16 ? 2 : 4;
    const size_t qstride = (size_t)Q * sh.H * D * es;
    const int nr4 = rows_total >= 16 ? 16 : ((rows_total + 3) & ~3);
    const size_t lds = decode_smem_bytes(nr4, pl.cpw);
    hipError_t e = sh.dtype == VARRATE_BF16 ? set_smem_attr<false>(lds) : set_smem_attr<true>(lds);
    if (e != hipSuccess) return e;
    for (int s0 = 0; s0 < S; s0 += DC_SEQ) {
        const int ns = S - s0 < DC_SEQ ? S - s0 : DC_SEQ;
        DecParams prm;
        for (int i = 0; i < ns; ++i) {
            const varrate_cache& c = caches[s0 + i];
            prm.seq[i] = DecSeq{c.coef_k, c.coef_v, c.srank, c.chunk_off, c.k_exact, c.v_exact,
                                (const uint8_t*)q + (s0 + i) * qstride, (uint8_t*)out + (s0 + i) * qstride,
                                c.n_exact};
        }
        for (int i = ns; i < DC_SEQ; ++i) prm.seq[i] = prm.seq[0];
        prm.PK = PK;
        prm.PV = PV;
        prm.part = part + (size_t)s0 * sh.G * pl.nqt * (pl.n_wg + 1) * DC_REC;
        prm.N = sh.n - sh.w;
        prm.coef_stride = caches[s0].coef_stride;
        prm.cap = caches[s0].cap;
        prm.G = sh.G;
        prm.H = sh.H;
        prm.hpg = hpg;
        prm.nqt = pl.nqt;
        prm.rows_total = rows_total;
        prm.n_chunks = pl.n_chunks;
        prm.cpw = pl.cpw;
        prm.n_wg = pl.n_wg;
        prm.tpw = pl.tpw;
        prm.total_tiles = pl.total_tiles;
        dim3 grid(pl.n_wg + 1, sh.G * pl.nqt, ns);
        if (sh.dtype == VARRATE_BF16) decode_kernel<false><<<grid, DC_THREADS, lds, st>>>(prm);
        else decode_kernel<true><<<grid, DC_THREADS, lds, st>>>(prm);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        MergeParams mp;
        mp.part = prm.part;
        mp.PV = PV;
        mp.out = (uint8_t*)out + s0 * qstride;
        mp.out_seq_stride = (int64_t)Q * sh.H * D;
        mp.G = sh.G;
        mp.H = sh.H;
        mp.hpg = hpg;
        mp.nqt = pl.nqt;
        mp.rows_total = rows_total;
        mp.n_wg = pl.n_wg;
        const unsigned nunits = (unsigned)(ns * sh.G * pl.nqt);
        if (sh.dtype == VARRATE_BF16) decode_merge_kernel<false><<<nunits, DC_THREADS, 0, st>>>(mp);
        else decode_merge_kernel<true><<<nunits, DC_THREADS, 0, st>>>(mp);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace vr
