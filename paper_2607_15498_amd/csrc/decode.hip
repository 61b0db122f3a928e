// Rank-space decode attention over the compressed cache, gfx950.
//
// Attention over the reconstructed cache of Eq. (6) without reconstructing it: with an
// orthonormal key basis <q, P_K^T (m . c)> = <P_K q, m . c>, and the value side is linear,
// so  o = P_V^T (sum_t p_t m_t . c^V_t) + sum_e p_e v_e.
//
// Grid (n_wg + 1, G * nqt, S).  Workgroup x < n_wg streams chunks [x cpw, (x+1) cpw) of KV
// head g for one sequence and one tile of up to 16 query rows (row = query * H/G + head);
// workgroup x == n_wg attends to the exact slots (window + appended tokens) in the
// original space.  Per workgroup (8 waves):
//   1. q' = P_K[g] q / sqrt(d) by MFMA (basis split into bf16 hi + lo parts, ~2^-16 error);
//   2. waves take 32-token tiles of the rank-sorted storage.  Each lane gathers its MFMA
//      operands straight from the packed ragged rows: 16-byte row segments for the score
//      tile (tokens x coefficients, masked past each token's rank) and, for the value
//      tile, the coefficients of 8 tokens at one rank index.  Scores, an online softmax
//      whose C-fragment layout already is the next A-fragment layout (no shuffles), and a
//      rank-space accumulation acc[row][j] += p c^V (p split into hi + lo bf16 parts);
//   3. the waves' (max, sum, acc) are combined in a fixed order and written as one partial;
//   4. the last workgroup to finish for (sequence, head, row tile) merges all partials by
//      log-sum-exp, rotates the rank-space sum back with P_V^T and adds the exact part.
// Tiles of a chunk are stored rank-descending, so a tile's first token bounds the MFMA
// steps (ceil(r_max/32) score steps, ceil(r_max/16) value blocks).
#include "vr_internal.h"

namespace vr {

constexpr int DC_THREADS = 512;
constexpr int DC_WAVES = 8;
constexpr int DC_SEQ = 16;           // sequences per launch
constexpr int DC_REC = 16 + 16 + 16 * D;   // floats per partial record: m, l, acc[16][128]
constexpr int DC_MAX_CPW = 16;

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
    uint32_t* counters;
    int64_t N, coef_stride, cap;
    int G, H, hpg, nqt, rows_total, n_chunks, cpw, n_wg;
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

template <bool F32>
__global__ __launch_bounds__(DC_THREADS) void decode_kernel(DecParams p) {
    typedef typename Elem<F32>::T ET;
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    const int x = blockIdx.x, gq = blockIdx.y, sq = blockIdx.z;
    const int g = gq / p.nqt, qt = gq % p.nqt;
    const DecSeq S = p.seq[sq];
    const int rows = min(16, p.rows_total - 16 * qt);
    const int nr4 = (rows + 3) & ~3;
    const bool exact = x == p.n_wg;
    const int cpw = p.cpw;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int grp = lane >> 4, col = lane & 15;

    float* qp = reinterpret_cast<float*>(smem);                 // [16][128]
    float* comb = qp + 16 * D;                                  // [4][nr4][128]
    float* cm = comb + 4 * nr4 * D;                             // [8][16]
    float* cl = cm + DC_WAVES * 16;                             // [8][16]
    float* mrow = cl + DC_WAVES * 16;                           // [16]
    float* lrow = mrow + 16;                                    // [16]
    uint32_t* cb = reinterpret_cast<uint32_t*>(lrow + 16);      // [cpw]
    int* cT = reinterpret_cast<int*>(cb + DC_MAX_CPW);          // [cpw]
    int* ctile = cT + DC_MAX_CPW;                               // [cpw + 1]
    int* flag = ctile + DC_MAX_CPW + 1;
    uint16_t* so = reinterpret_cast<uint16_t*>(flag + 3);       // [cpw][256]
    uint8_t* sr = reinterpret_cast<uint8_t*>(so + cpw * CHUNK); // [cpw][256]

    const float scale = 0.08838834764831845f;  // 1/sqrt(128)
    const ET* qsrc = reinterpret_cast<const ET*>(S.q);

    // ---- 1. query rows into LDS: rotated into the key basis (coded) or as is (exact)
    if (!exact) {
        const float* P = p.PK + (int64_t)g * D * D;
        const int qrow = 16 * qt + col;
        const bool ok = qrow < p.rows_total;
        const int query = ok ? qrow / p.hpg : 0, hh = ok ? qrow % p.hpg : 0;
        const ET* qv = qsrc + ((int64_t)query * p.H + g * p.hpg + hh) * D;
        f32x4 c = {0, 0, 0, 0};
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int c0 = 32 * s + 8 * grp;
            float a8[8];
            const float* src = P + (16 * wave + col) * D + c0;
            u32x4 a0 = load16(src), a1 = load16(src + 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) { a8[e] = __uint_as_float(a0[e]); a8[4 + e] = __uint_as_float(a1[e]); }
            u32x4 ah, al, bh, bl;
            split8(a8, ah, al);
            load_row8<F32>(qv + c0, ok ? 8 : 0, bh, bl);
            c = mfma(ah, bh, c);
            c = mfma(al, bh, c);
            if constexpr (F32) c = mfma(ah, bl, c);
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) qp[col * D + 16 * wave + 4 * grp + v] = c[v] * scale;
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
            qp[idx] = val * scale;
        }
    }
    // ---- chunk metadata
    if (!exact) {
        for (int cc = 0; cc < cpw; ++cc) {
            const int c = x * cpw + cc;
            const int64_t t0 = (int64_t)c * CHUNK;
            const int T = c < p.n_chunks ? (int)((p.N - t0) < CHUNK ? (p.N - t0) : CHUNK) : 0;
            if (tid == 0) { cT[cc] = T; cb[cc] = c < p.n_chunks ? S.chunk_off[c] : 0; }
            for (int i = tid; i < CHUNK; i += DC_THREADS) sr[cc * CHUNK + i] = i < T ? S.srank[t0 + i] : 0;
        }
    }
    __syncthreads();
    if (!exact) {
        for (int cc = wave; cc < cpw; cc += DC_WAVES) {
            uint32_t r[4], loc = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e) { r[e] = sr[cc * CHUNK + 4 * lane + e]; loc += r[e]; }
            uint32_t xs = loc;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                uint32_t y = __shfl_up(xs, off, 64);
                if (lane >= off) xs += y;
            }
            uint32_t pre = xs - loc;
#pragma unroll
            for (int e = 0; e < 4; ++e) { so[cc * CHUNK + 4 * lane + e] = (uint16_t)pre; pre += r[e]; }
        }
        if (tid == 0) {
            int acc = 0;
            for (int cc = 0; cc < cpw; ++cc) { ctile[cc] = acc; acc += (cT[cc] + 31) / 32; }
            ctile[cpw] = acc;
        }
    } else if (tid == 0) {
        ctile[0] = 0;
        ctile[1] = (int)((S.n_exact + 31) / 32);
    }
    __syncthreads();

    // ---- 2. score-operand fragments of this wave: lane -> query row col, K group grp
    u32x4 qh[4], ql[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        float v8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v8[e] = qp[col * D + 32 * s + 8 * grp + e];
        split8(v8, qh[s], ql[s]);
    }

    const int ntiles = exact ? ctile[1] : ctile[cpw];
    const ET* kbase_all = reinterpret_cast<const ET*>(exact ? S.k_exact : S.coef_k);
    const ET* vbase_all = reinterpret_cast<const ET*>(exact ? S.v_exact : S.coef_v);
    float m_run = -INFINITY, l_part = 0.f;
    f32x4 acc[8];
#pragma unroll
    for (int b = 0; b < 8; ++b) acc[b] = f32x4{0, 0, 0, 0};

    for (int tile = wave; tile < ntiles; tile += DC_WAVES) {
        int cc = 0, i0, T, rmax;
        int64_t base;
        if (exact) {
            i0 = tile * 32;
            T = (int)S.n_exact;
            rmax = D;
            base = (int64_t)g * p.cap * D;
        } else {
            while (tile >= ctile[cc + 1]) ++cc;
            i0 = (tile - ctile[cc]) * 32;
            T = cT[cc];
            rmax = sr[cc * CHUNK + i0];
            base = (int64_t)g * p.coef_stride + cb[cc];
        }
        const ET* Kb = kbase_all + base;
        const ET* Vb = vbase_all + base;
        const int ks = (rmax + 31) >> 5, nb = (rmax + 15) >> 4;
        auto meta = [&](int i, int& r, int& o) {
            if (i >= T) { r = 0; o = 0; return; }
            if (exact) { r = D; o = i * D; }
            else { r = sr[cc * CHUNK + i]; o = so[cc * CHUNK + i]; }
        };
        // score operands: rows = tokens i0 + 16a + col
        u32x4 kh[2][4], kl[2][4];
#pragma unroll
        for (int a = 0; a < 2; ++a) {
            int r, o;
            meta(i0 + 16 * a + col, r, o);
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                if (s < ks) {
                    const int c0 = 32 * s + 8 * grp;
                    int nv = r - c0;
                    nv = nv < 0 ? 0 : (nv > 8 ? 8 : nv);
                    load_row8<F32>(Kb + o + c0, nv, kh[a][s], kl[a][s]);
                } else {
                    kh[a][s] = kl[a][s] = u32x4{0, 0, 0, 0};
                }
            }
        }
        // value operands: K slot e <-> token i0 + 16 (e / 4) + 4 grp + (e % 4)
        int vr_[8], vo_[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) meta(i0 + 16 * (e >> 2) + 4 * grp + (e & 3), vr_[e], vo_[e]);
        u32x4 vh[8], vl[8];
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            if (b < nb) {
                const int j = 16 * b + col;
                float f8[8];
                uint32_t h16[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    if constexpr (F32) f8[e] = j < vr_[e] ? Vb[vo_[e] + j] : 0.f;
                    else h16[e] = j < vr_[e] ? (uint32_t)Vb[vo_[e] + j] : 0u;
                }
                if constexpr (F32) {
                    split8(f8, vh[b], vl[b]);
                } else {
#pragma unroll
                    for (int k = 0; k < 4; ++k) vh[b][k] = pack2(h16[2 * k], h16[2 * k + 1]);
                    vl[b] = u32x4{0, 0, 0, 0};
                }
            } else {
                vh[b] = vl[b] = u32x4{0, 0, 0, 0};
            }
        }
        // scores: C lane -> query row col, tokens i0 + 16a + 4grp + v
        f32x4 sc[2];
#pragma unroll
        for (int a = 0; a < 2; ++a) {
            f32x4 c = {0, 0, 0, 0};
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                if (s < ks) {
                    c = mfma(kh[a][s], qh[s], c);
                    c = mfma(kh[a][s], ql[s], c);
                    if constexpr (F32) c = mfma(kl[a][s], qh[s], c);
                }
            }
            sc[a] = c;
        }
        float sv[8];
        float tmax = -INFINITY;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int slot = i0 + 16 * (e >> 2) + 4 * grp + (e & 3);
            sv[e] = slot < T ? sc[e >> 2][e & 3] : -INFINITY;
            tmax = fmaxf(tmax, sv[e]);
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
        float pv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            pv[e] = m_run == -INFINITY ? 0.f : fast_exp(sv[e] - m_run);
            l_part += pv[e];
        }
        u32x4 ph, pl;
        split8(pv, ph, pl);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            if (b < nb) {
                acc[b] = mfma(ph, vh[b], acc[b]);
                acc[b] = mfma(pl, vh[b], acc[b]);
                if constexpr (F32) acc[b] = mfma(ph, vl[b], acc[b]);
            }
        }
    }

    // ---- 3. combine the waves of this workgroup (fixed order)
    float lsum = l_part + shfl_xor_f(l_part, 16);
    lsum += shfl_xor_f(lsum, 32);
    if (lane < 16) { cm[wave * 16 + col] = m_run; cl[wave * 16 + col] = lsum; }
    __syncthreads();
    if (tid < 16) {
        float M = -INFINITY;
        for (int w = 0; w < DC_WAVES; ++w) M = fmaxf(M, cm[w * 16 + tid]);
        float L = 0.f;
        for (int w = 0; w < DC_WAVES; ++w) {
            const float mw = cm[w * 16 + tid];
            L += mw == -INFINITY ? 0.f : cl[w * 16 + tid] * fast_exp(mw - M);
        }
        mrow[tid] = M;
        lrow[tid] = L;
    }
    __syncthreads();
    float fac[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const int row = 4 * grp + v;
        const float mw = cm[wave * 16 + row];
        fac[v] = mw == -INFINITY ? 0.f : fast_exp(mw - mrow[row]);
    }
    if (wave >= 4) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int row = 4 * grp + v;
            if (row < nr4) {
#pragma unroll
                for (int b = 0; b < 8; ++b) comb[((wave - 4) * nr4 + row) * D + 16 * b + col] = acc[b][v] * fac[v];
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
                    float* dst = &comb[(wave * nr4 + row) * D + 16 * b + col];
                    *dst = acc[b][v] * fac[v] + *dst;
                }
            }
        }
    }
    __syncthreads();
    const int units = p.G * p.nqt;
    float* rec = p.part + (((int64_t)sq * units + gq) * (p.n_wg + 1) + x) * DC_REC;
    for (int idx = tid; idx < nr4 * D; idx += DC_THREADS) {
        const float v = ((comb[idx] + comb[nr4 * D + idx]) + comb[2 * nr4 * D + idx]) + comb[3 * nr4 * D + idx];
        rec[32 + idx] = v;
    }
    if (tid < 16) { rec[tid] = mrow[tid]; rec[16 + tid] = lrow[tid]; }

    // ---- 4. last workgroup of (sequence, head, row tile) merges
    __threadfence();
    __syncthreads();
    uint32_t* ctr = p.counters + (int64_t)sq * units + gq;
    if (tid == 0) flag[0] = atomicAdd(ctr, 1u) == (uint32_t)p.n_wg;
    __syncthreads();
    if (!flag[0]) return;
    __threadfence();
    const int nrec = p.n_wg + 1;
    const float* recs = p.part + (((int64_t)sq * units + gq) * nrec) * DC_REC;
    if (tid < 16) {
        float M = -INFINITY;
        for (int r = 0; r < nrec; ++r) M = fmaxf(M, __builtin_nontemporal_load(&recs[(int64_t)r * DC_REC + tid]));
        float L = 0.f;
        for (int r = 0; r < nrec; ++r) {
            const float mr = __builtin_nontemporal_load(&recs[(int64_t)r * DC_REC + tid]);
            if (mr != -INFINITY) L += __builtin_nontemporal_load(&recs[(int64_t)r * DC_REC + 16 + tid]) * fast_exp(mr - M);
        }
        mrow[tid] = M;
        lrow[tid] = L;
    }
    __syncthreads();
    float* accR = comb;             // [nr4][128] rank-space sum
    float* accE = comb + nr4 * D;   // [nr4][128] exact-slot sum (original space)
    for (int idx = tid; idx < nr4 * D; idx += DC_THREADS) {
        const int row = idx / D;
        const float M = mrow[row];
        float sR = 0.f;
        for (int r = 0; r < p.n_wg; ++r) {
            const float mr = __builtin_nontemporal_load(&recs[(int64_t)r * DC_REC + row]);
            if (mr != -INFINITY) sR += fast_exp(mr - M) * __builtin_nontemporal_load(&recs[(int64_t)r * DC_REC + 32 + idx]);
        }
        const float me = __builtin_nontemporal_load(&recs[(int64_t)p.n_wg * DC_REC + row]);
        const float sE = me == -INFINITY ? 0.f
                         : fast_exp(me - M) * __builtin_nontemporal_load(&recs[(int64_t)p.n_wg * DC_REC + 32 + idx]);
        accR[idx] = sR;
        accE[idx] = sE;
    }
    __syncthreads();
    // back-rotation o = P_V^T accR + accE, divided by L: thread -> (column c, rows rg + 4k)
    {
        const int c = tid & (D - 1), rg = tid >> 7;
        const float* PV = p.PV + (int64_t)g * D * D;
        float o[4] = {0.f, 0.f, 0.f, 0.f};
        for (int j = 0; j < D; ++j) {
            const float pvj = PV[j * D + c];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int row = rg + 4 * k;
                if (row < rows) o[k] += pvj * accR[row * D + j];
            }
        }
        ET* out = reinterpret_cast<ET*>(S.out);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int row = rg + 4 * k;
            if (row < rows) {
                const float val = (o[k] + accE[row * D + c]) / lrow[row];
                const int qrow = 16 * qt + row;
                const int query = qrow / p.hpg, hh = qrow % p.hpg;
                const int64_t oi = ((int64_t)query * p.H + g * p.hpg + hh) * D + c;
                if constexpr (F32) out[oi] = val;
                else out[oi] = (uint16_t)f32_to_bf16(val);
            }
        }
    }
    if (tid == 0) *ctr = 0u;
}

// ----------------------------------------------------------------------------------------
struct DecPlan {
    int nqt, n_chunks, cpw, n_wg;
};

static DecPlan plan_decode(const varrate_shape& sh, int S, int Q) {
    DecPlan pl;
    const int64_t N = sh.n - sh.w;
    const int rows_total = Q * (sh.H / sh.G);
    pl.nqt = (rows_total + 15) / 16;
    pl.n_chunks = (int)((N + CHUNK - 1) / CHUNK);
    const int units = (S < DC_SEQ ? S : DC_SEQ) * sh.G * pl.nqt;
    int target = 256 / (units > 0 ? units : 1);
    if (target < 1) target = 1;
    int cpw = (pl.n_chunks + target - 1) / target;
    cpw = cpw < 1 ? 1 : (cpw > DC_MAX_CPW ? DC_MAX_CPW : cpw);
    pl.cpw = cpw;
    pl.n_wg = (pl.n_chunks + cpw - 1) / cpw;
    return pl;
}

static size_t decode_lds_bytes(int nr4, int cpw) {
    return (size_t)(16 * D + 4 * nr4 * D + 2 * DC_WAVES * 16 + 32) * 4 +
           (size_t)(3 * DC_MAX_CPW + 4) * 4 + (size_t)cpw * CHUNK * 3 + 64;
}

// Workspace: a fixed counter region first (each merge resets its own counter, and no
// call ever writes partials there, so a workspace zero-filled once stays valid for any
// shape), then the partial records.
constexpr size_t DC_COUNTERS = 16384;

size_t decode_units(const varrate_shape& sh, int S, int Q) {
    return (size_t)S * sh.G * plan_decode(sh, S, Q).nqt;
}

size_t decode_ws_bytes(const varrate_shape& sh, int S, int Q) {
    DecPlan pl = plan_decode(sh, S, Q);
    const size_t units = (size_t)S * sh.G * pl.nqt;
    return DC_COUNTERS * sizeof(uint32_t) + align256(units * (pl.n_wg + 1) * DC_REC * sizeof(float));
}

hipError_t launch_decode(const varrate_shape& sh, const varrate_cache* caches, int S, const void* q,
                         int Q, const float* PK, const float* PV, void* out, uint8_t* ws,
                         hipStream_t st) {
    DecPlan pl = plan_decode(sh, S, Q);
    const int hpg = sh.H / sh.G;
    const int rows_total = Q * hpg;
    const size_t units_all = (size_t)S * sh.G * pl.nqt;
    if (units_all > DC_COUNTERS) return hipErrorInvalidValue;
    uint32_t* counters = (uint32_t*)ws;
    float* part = (float*)(ws + DC_COUNTERS * sizeof(uint32_t));
    const size_t es = sh.dtype == VARRATE_BF16 ? 2 : 4;
    const size_t qstride = (size_t)Q * sh.H * D * es;
    const int nr4 = rows_total >= 16 ? 16 : ((rows_total + 3) & ~3);
    const size_t lds = decode_lds_bytes(nr4, pl.cpw);
    const void* fn = sh.dtype == VARRATE_BF16 ? (const void*)decode_kernel<false> : (const void*)decode_kernel<true>;
    hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
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
        prm.counters = counters + (size_t)s0 * sh.G * pl.nqt;
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
        dim3 grid(pl.n_wg + 1, sh.G * pl.nqt, ns);
        if (sh.dtype == VARRATE_BF16) decode_kernel<false><<<grid, DC_THREADS, lds, st>>>(prm);
        else decode_kernel<true><<<grid, DC_THREADS, lds, st>>>(prm);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace vr
