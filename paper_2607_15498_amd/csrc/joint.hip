// Shared cross-head basis (Sec. 3.1 Eq. (1) "Joint per-token vector" and "Shared basis";
// Eq. (3) in joint units; Eq. (6)), gfx950.
//
// A token's keys and values of all G heads form z_t = [k_t; v_t] (Dz = 2 G d entries), coded
// against one basis W [R][Dz]: c_t = W z_t truncated to its rank, one coefficient row for
// every head and both K and V, stored in original token order (token t's row at offset[t]).
//
// Compress: the salience and allocation passes of the per-head codec (cap R, 16-bit ranks,
// per-token offsets), then jproj_kernel: C = Z W^T by bf16 MFMA (W split into bf16 hi + lo
// parts, Z exact in bf16), a workgroup per (256 tokens, 128 coefficients), skipped when no
// token of the 256 reaches its coefficients.
//
// Decode (q [S][Q][H][d], rows = Q H <= 32 per sequence):
//   jq_kernel   q'_row = W_K,g q_row / sqrt(d) for every query row (fp32, [S][32][R]);
//   jd_kernel   streams 16-token tiles of the coefficient rows (original order) through LDS;
//               wave w owns coefficients [w R/8, (w + 1) R/8): it forms the partial scores of
//               its slice by MFMA (A = the tile's rows, B = q' fragments, bf16 hi + lo), the 8
//               partials are summed through LDS in a fixed order so every wave holds the same
//               scores and runs the same online softmax, and each wave accumulates the
//               rank-space value sum of its own slice (16x16x16 MFMA, the score fragment as
//               B operand).  One record (m, l, acc[32][R]) per workgroup;
//   jx_kernel   the exact rows (window and appended tokens) per query row, original space;
//   jm1_kernel  log-sum-exp combination of the records per (row, 64 coefficients);
//   jm2_kernel_part  rotation back with W_V,g^T for all of head g's rows: a workgroup per
//               (g, 32 output coordinates, 256 coefficients), 8 partial sums each;
//   jm2_kernel  the partial sums added in order, the exact part added, division by the sum.
#include <type_traits>

#include "vr_internal.h"

namespace vr {

typedef short j_s16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t j_u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f32x4 jmfma16(j_u32x2 a, j_u32x2 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(j_s16x4, a), __builtin_bit_cast(j_s16x4, b),
                                                     c, 0, 0, 0);
}

// 8 consecutive bf16 at element index a of an LDS array (any 2-byte alignment)
__device__ __forceinline__ u32x4 j_row8(const uint32_t* w, int a) {
    const int w0 = a >> 1;
    const uint32_t sh = (uint32_t)(a & 1) * 16u;
    const uint32_t d0 = w[w0], d1 = w[w0 + 1], d2 = w[w0 + 2], d3 = w[w0 + 3], d4 = w[w0 + 4];
    return u32x4{__builtin_amdgcn_alignbit(d1, d0, sh), __builtin_amdgcn_alignbit(d2, d1, sh),
                 __builtin_amdgcn_alignbit(d3, d2, sh), __builtin_amdgcn_alignbit(d4, d3, sh)};
}

// 4 fp32 -> bf16x4 hi and lo parts
__device__ __forceinline__ void j_split4(const float* x, j_u32x2& hi, j_u32x2& lo) {
    uint32_t h0, l0, h1, l1;
    split2(x[0], x[1], h0, l0);
    split2(x[2], x[3], h1, l1);
    hi = j_u32x2{h0, h1};
    lo = j_u32x2{l0, l1};
}

// the first nv of 8 bf16 elements kept
__device__ __forceinline__ u32x4 j_keep(u32x4 x, int nv) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t m = nv >= 2 * k + 2 ? 0xFFFFFFFFu : (nv == 2 * k + 1 ? 0x0000FFFFu : 0u);
        x[k] &= m;
    }
    return x;
}

// ---- projection ---------------------------------------------------------------------------
constexpr int JP_T = 512;
constexpr int JP_TOK = 256;      // tokens per workgroup: 32 per wave (two 16-token blocks)
constexpr int JP_COL = 128;      // coefficients per workgroup: 8 blocks of 16

template <bool F32>
__global__ __launch_bounds__(JP_T, 2) void jproj_kernel(const void* __restrict__ Kv, const void* __restrict__ Vv,
                                                        const float* __restrict__ W,
                                                        const uint16_t* __restrict__ rank,
                                                        const uint32_t* __restrict__ offset, void* __restrict__ coefv,
                                                        int64_t N, int G, int R) {
    typedef typename std::conditional<F32, float, uint16_t>::type ET;
    __shared__ __attribute__((aligned(16))) u32x4 wl[2][2][8][64];   // [buffer][hi, lo][block][lane]
    __shared__ uint32_t s_max;
    const ET* K = reinterpret_cast<const ET*>(Kv);
    const ET* V = reinterpret_cast<const ET*>(Vv);
    ET* coef = reinterpret_cast<ET*>(coefv);
    const int half = G * D, Dz = 2 * G * D;
    const int nb = R / JP_COL;
    const int tb = blockIdx.x / nb, cb = blockIdx.x % nb;
    const int64_t t_base = (int64_t)tb * JP_TOK;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, col = lane & 15, grp = lane >> 4;
    // skip the workgroup when no token of its 256 keeps any of its 128 coefficients
    if (tid == 0) s_max = 0u;
    __syncthreads();
    if (tid < JP_TOK && t_base + tid < N) atomicMax(&s_max, (uint32_t)rank[t_base + tid]);
    __syncthreads();
    const int j_base = cb * JP_COL;
    if ((int)s_max <= j_base) return;
    // this wave's tokens: t_base + 32 wave + 16 mb + col (A rows); the stores' tokens below
    int64_t ta[2];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
        const int64_t t = t_base + 32 * wave + 16 * mb + col;
        ta[mb] = t < N ? t : N - 1;
    }
    // W staging: thread -> (block tid >> 6, lane): coefficient j_base + 16 (tid >> 6) + (lane & 15),
    // z coordinates k0 + 8 grp .. + 7
    const float* wrow = W + (int64_t)(j_base + 16 * (tid >> 6) + col) * Dz + 8 * grp;
    auto load_w = [&](int k0, u32x4& a, u32x4& b) {
        a = load16(wrow + k0);
        b = load16(wrow + k0 + 4);
    };
    auto put_w = [&](int buf, const u32x4& a, const u32x4& b) {
        float x8[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) { x8[e] = __uint_as_float(a[e]); x8[4 + e] = __uint_as_float(b[e]); }
        u32x4 h, l;
        split8(x8, h, l);
        wl[buf][0][tid >> 6][lane] = h;
        wl[buf][1][tid >> 6][lane] = l;
    };
    // A fragments (z of the wave's tokens): bf16 as 8 raw elements; fp32 as two 16-byte pieces
    auto zsrc = [&](int64_t t, int k) -> const ET* {
        return k < half ? K + t * half + k : V + t * half + (k - half);
    };
    u32x4 za[2][2];
    auto load_z = [&](int k0, u32x4 (&z)[2][2]) {
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
            const ET* p = zsrc(ta[mb], k0 + 8 * grp);
            if constexpr (F32) { z[mb][0] = load16(p); z[mb][1] = load16(p + 4); }
            else { z[mb][0] = load16(p); z[mb][1] = u32x4{0, 0, 0, 0}; }
        }
    };
    f32x4 acc[2][8];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int b = 0; b < 8; ++b) acc[mb][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int nsteps = Dz / 32;
    u32x4 wa, wb;
    load_w(0, wa, wb);
    load_z(0, za);
    put_w(0, wa, wb);
    for (int s = 0; s < nsteps; ++s) {
        __syncthreads();    // buffer s & 1 is written; every wave is done with buffer (s + 1) & 1
        u32x4 zn[2][2];
        const bool more = s + 1 < nsteps;
        if (more) {
            load_w(32 * (s + 1), wa, wb);
            load_z(32 * (s + 1), zn);
        }
        const int buf = s & 1;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
            u32x4 ah, al;
            if constexpr (F32) {
                float x8[8];
#pragma unroll
                for (int e = 0; e < 4; ++e) { x8[e] = __uint_as_float(za[mb][0][e]); x8[4 + e] = __uint_as_float(za[mb][1][e]); }
                split8(x8, ah, al);
            } else {
                ah = za[mb][0];
            }
#pragma unroll
            for (int b = 0; b < 8; ++b) {
                const u32x4 wh = wl[buf][0][b][lane], wlo = wl[buf][1][b][lane];
                acc[mb][b] = mfma(ah, wh, acc[mb][b]);
                acc[mb][b] = mfma(ah, wlo, acc[mb][b]);
                if constexpr (F32) acc[mb][b] = mfma(al, wh, acc[mb][b]);
            }
        }
        if (more) {
            put_w(buf ^ 1, wa, wb);
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) { za[mb][0] = zn[mb][0]; za[mb][1] = zn[mb][1]; }
        }
    }
    // C lane -> tokens 4 grp + v of block mb, coefficient j_base + 16 b + col
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int64_t t = t_base + 32 * wave + 16 * mb + 4 * grp + v;
            if (t >= N) continue;
            const int r = rank[t];
            const uint32_t o = offset[t];
#pragma unroll
            for (int b = 0; b < 8; ++b) {
                const int j = j_base + 16 * b + col;
                if (j < r) coef[o + j] = to_elem<ET>(acc[mb][b][v]);
            }
        }
    }
}

hipError_t launch_joint_project(const varrate_shape& sh, int R, const void* K, const void* V, const float* W,
                                const uint16_t* rank, const uint32_t* offset, void* coef, hipStream_t st) {
    const int64_t N = sh.n - sh.w;
    const unsigned blocks = (unsigned)(((N + JP_TOK - 1) / JP_TOK) * (R / JP_COL));
    if (sh.dtype == VARRATE_BF16)
        jproj_kernel<false><<<blocks, JP_T, 0, st>>>(K, V, W, rank, offset, coef, N, sh.G, R);
    else
        jproj_kernel<true><<<blocks, JP_T, 0, st>>>(K, V, W, rank, offset, coef, N, sh.G, R);
    return hipGetLastError();
}

// ---- decode ---------------------------------------------------------------------------------
constexpr int JW = 8;                 // waves per decode workgroup
constexpr int JD_T = 64 * JW;
constexpr int JSEQ = 16;              // sequences per launch
constexpr int JROWS = 32;             // query rows per sequence (two 16-row tiles)
constexpr int JREC_HEAD = 2 * JROWS;  // m[32], l[32] before acc[32][R]
constexpr int JX_CAP = 8192;          // exact slots the exact kernel holds in LDS

struct JSeq {
    const void* coef;
    const uint16_t* rank;
    const uint32_t* offset;
    const void* kx;
    const void* vx;
    const void* q;
    void* out;
    int64_t n_exact;
};

struct JDec {
    JSeq seq[JSEQ];
    const float* W;
    float* qp;      // [seq][32][R] q' (scaled by 1/sqrt(d))
    float* rec;     // [seq][n_wg][JREC_HEAD + 32 R]
    float* xrec;    // [seq][32][2 + 128]: m, l, acc of the exact rows
    float* comb;    // [seq][32][R] combined rank-space sums
    float* ml;      // [seq][32][2] M, L
    int64_t N, cap;
    int G, H, hpg, rows, R, n_wg, tpw, total_tiles;
};

// q'[s][row][k] = (1/sqrt(d)) sum_i W[k][g d + i] q[s][row][i]; rows past the query rows are 0.
// Workgroup per (sequence, row, 64 coefficients): 4 threads per coefficient, 32 dims each.
template <bool F32>
__global__ __launch_bounds__(256) void jq_kernel(JDec p) {
    typedef typename std::conditional<F32, float, uint16_t>::type ET;
    const int kb_n = p.R / 64;
    const int s = blockIdx.x / (JROWS * kb_n), rem = blockIdx.x % (JROWS * kb_n);
    const int row = rem / kb_n, kb = rem % kb_n;
    const int k = kb * 64 + (threadIdx.x >> 2), qd = threadIdx.x & 3;
    float acc = 0.f;
    if (row < p.rows) {
        const int h = row % p.H, query = row / p.H, g = h / p.hpg;
        const ET* q = reinterpret_cast<const ET*>(p.seq[s].q) + ((int64_t)query * p.H + h) * D;
        const float* w = p.W + (int64_t)k * (2 * p.G * D) + g * D;
        for (int i = 32 * qd; i < 32 * qd + 32; ++i) acc = fmaf(w[i], elem_f(q[i]), acc);
    }
    acc += __shfl_xor(acc, 1, 64);
    acc += __shfl_xor(acc, 2, 64);
    if (qd == 0) p.qp[((int64_t)s * JROWS + row) * p.R + k] = acc * 0.08838834764831845f;
}

// LDS of the decode workgroup
constexpr int JD_STAGE = 16 * 1024 * 2 + 64;   // bytes: 16 tokens x 1024 bf16 + over-read slack

template <bool F32, int RT>
__global__ __launch_bounds__(JD_T, 2) void jd_kernel(JDec p) {
    typedef typename std::conditional<F32, float, uint16_t>::type ET;
    constexpr int EPU = 16 / (int)sizeof(ET);
    __shared__ __attribute__((aligned(16))) uint8_t stage_b[F32 ? 2 * JD_STAGE : JD_STAGE];
    __shared__ __attribute__((aligned(16))) f32x4 psc[JW][RT][64];
    __shared__ int to_s[17];
    const ET* stage = reinterpret_cast<const ET*>(stage_b);
    const int s = blockIdx.x / p.n_wg, x = blockIdx.x % p.n_wg;
    const JSeq& S = p.seq[s];
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, col = lane & 15, grp = lane >> 4;
    const int RS = p.R / JW, kss = RS / 32, nvb = RS / 16;
    const int slice = wave * RS;
    const ET* coef = reinterpret_cast<const ET*>(S.coef);
    // q' fragments of this wave's slice: lane -> row 16 rt + col, coefficients slice + 32 st +
    // 8 grp .. + 7, bf16 hi and lo
    u32x4 qf[RT][4][2];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            qf[rt][st][0] = qf[rt][st][1] = u32x4{0, 0, 0, 0};
            if (st < kss) {
                const float* src = p.qp + ((int64_t)s * JROWS + 16 * rt + col) * p.R + slice + 32 * st + 8 * grp;
                const u32x4 a = load16(src), b = load16(src + 4);
                float x8[8];
#pragma unroll
                for (int e = 0; e < 4; ++e) { x8[e] = __uint_as_float(a[e]); x8[4 + e] = __uint_as_float(b[e]); }
                split8(x8, qf[rt][st][0], qf[rt][st][1]);
            }
        }
    }
    f32x4 acc[RT][8];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int b = 0; b < 8; ++b) acc[rt][b] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run[RT], l_part[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) { m_run[rt] = -INFINITY; l_part[rt] = 0.f; }

    const int tau0 = x * p.tpw, tau1 = min(tau0 + p.tpw, p.total_tiles);
    // stage of one tile: elements [s0, s0 + EPU u) with s0 = offset[16 tau] rounded down to EPU;
    // thread tid moves units tid + 512 i (at most 16 R / EPU + 2 units)
    constexpr int NU = F32 ? 9 : 5;    // 16 x 1024 elements: 2050 units (bf16), 4098 (fp32)
    u32x4 pre[NU];
    int pre_s0 = 0, pre_nu = 0;
    uint32_t pre_to = 0;
    auto fetch = [&](int tau) {
        const int64_t t0 = 16 * (int64_t)tau;
        const int64_t t1 = min(t0 + 16, p.N);
        const uint32_t b0 = S.offset[t0], b1 = S.offset[t1];
        pre_s0 = (int)(b0 & ~(uint32_t)(EPU - 1));
        pre_nu = (int)((b1 - (uint32_t)pre_s0 + EPU - 1) / EPU);
#pragma unroll
        for (int i = 0; i < NU; ++i) {
            const int u = tid + JD_T * i;
            pre[i] = u < pre_nu ? load16(coef + pre_s0 + (int64_t)EPU * u) : u32x4{0, 0, 0, 0};
        }
        // token offsets of the tile relative to s0 (tokens past N take the end)
        if (tid <= 16) pre_to = S.offset[min(t0 + tid, p.N)] - (uint32_t)pre_s0;
    };
    if (tau0 < tau1) fetch(tau0);
    for (int tau = tau0; tau < tau1; ++tau) {
        // ---- staged tile into LDS, then prefetch the next
#pragma unroll
        for (int i = 0; i < NU; ++i) {
            const int u = tid + JD_T * i;
            if (u < pre_nu) reinterpret_cast<u32x4*>(stage_b)[u] = pre[i];
        }
        if (tid <= 16) to_s[tid] = (int)pre_to;
        __syncthreads();
        const int T = (int)min((int64_t)16, p.N - 16 * (int64_t)tau);
        if (tau + 1 < tau1) fetch(tau + 1);
        // ---- partial scores of this wave's slice: A = rows of token col, B = q'
        const int a_col = to_s[col], r_col = col < T ? to_s[col + 1] - to_s[col] : 0;
        // the tile's largest rank (a max over the 16 lanes of a row, then wave-uniform)
        int m = r_col;
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) m = max(m, __shfl_xor(m, o, 64));
        m = __builtin_amdgcn_readfirstlane(m);
        f32x4 sc[RT];
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) sc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            if (st < kss && slice + 32 * st < m) {
                const int kk = slice + 32 * st + 8 * grp;
                int nv = r_col - kk;
                nv = nv < 0 ? 0 : (nv > 8 ? 8 : nv);
                const int a = nv > 0 ? a_col + kk : 0;
                u32x4 kh, kl;
                if constexpr (F32) {
                    float x8[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) { const float v = stage[a + e]; x8[e] = e < nv ? v : 0.f; }
                    split8(x8, kh, kl);
                } else {
                    kh = j_keep(j_row8(reinterpret_cast<const uint32_t*>(stage_b), a), nv);
                }
#pragma unroll
                for (int rt = 0; rt < RT; ++rt) {
                    sc[rt] = mfma(kh, qf[rt][st][0], sc[rt]);
                    sc[rt] = mfma(kh, qf[rt][st][1], sc[rt]);
                    if constexpr (F32) sc[rt] = mfma(kl, qf[rt][st][0], sc[rt]);
                }
            }
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) psc[wave][rt][lane] = sc[rt];
        __syncthreads();
        // ---- full scores (fixed order over the waves), online softmax, value sums of the slice
        int rr[4], ao[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int t = 4 * grp + e;
            rr[e] = t < T ? to_s[t + 1] - to_s[t] : 0;
            ao[e] = to_s[t < T ? t : 0];
        }
        // value operands of the slice (lane -> coordinate slice + 16 b + col, tokens 4 grp ..
        // 4 grp + 3), built once for every row tile
        j_u32x2 vop[8], vopl[8];
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            vop[b] = vopl[b] = j_u32x2{0u, 0u};
            if (b < nvb && slice + 16 * b < m) {
                const int j = slice + 16 * b + col;
                float v4[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const bool ok = j < rr[e];
                    const float v = elem_f(stage[ok ? ao[e] + j : 0]);
                    v4[e] = ok ? v : 0.f;
                }
                if constexpr (F32) j_split4(v4, vop[b], vopl[b]);
                else vop[b] = j_u32x2{cvt_bf16x2(v4[0], v4[1]), cvt_bf16x2(v4[2], v4[3])};
            }
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
            f32x4 sv = psc[0][rt][lane];
#pragma unroll
            for (int w = 1; w < JW; ++w) sv = sv + psc[w][rt][lane];
            float s4[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) s4[v] = 4 * grp + v < T ? sv[v] : -INFINITY;
            float tmax = fmaxf(fmaxf(s4[0], s4[1]), fmaxf(s4[2], s4[3]));
            tmax = xmax32(xmax16(tmax));
            if (tmax > m_run[rt] + 8.f) {        // lane-uniform per row: every lane of the row agrees
                const float alpha = fast_exp(m_run[rt] - tmax);
                l_part[rt] *= alpha;
#pragma unroll
                for (int b = 0; b < 8; ++b) acc[rt][b] = acc[rt][b] * alpha;
                m_run[rt] = tmax;
            }
            float pv[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                pv[v] = fast_exp(s4[v] - m_run[rt]);
                l_part[rt] += pv[v];
            }
            j_u32x2 ph, pl;
            if constexpr (F32) {
                j_split4(pv, ph, pl);
            } else {
                ph = j_u32x2{cvt_bf16x2(pv[0], pv[1]), cvt_bf16x2(pv[2], pv[3])};
                pl = j_u32x2{0u, 0u};
            }
#pragma unroll
            for (int b = 0; b < 8; ++b) {
                if (b < nvb && slice + 16 * b < m) {
                    acc[rt][b] = jmfma16(vop[b], ph, acc[rt][b]);
                    if constexpr (F32) {
                        acc[rt][b] = jmfma16(vop[b], pl, acc[rt][b]);
                        acc[rt][b] = jmfma16(vopl[b], ph, acc[rt][b]);
                    }
                }
            }
        }
        __syncthreads();   // the stage and the partial scores are reused by the next tile
    }
    // ---- record: m, l per row (every wave holds the same), acc of the wave's slice
    float* rec = p.rec + ((int64_t)s * p.n_wg + x) * (JREC_HEAD + (int64_t)JROWS * p.R);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
        const float l = xsum32(xsum16(l_part[rt]));
        if (wave == 0 && lane < 16) {
            rec[16 * rt + col] = m_run[rt];
            rec[JROWS + 16 * rt + col] = l;
        }
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            if (b < nvb) {
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    rec[JREC_HEAD + (int64_t)(16 * rt + col) * p.R + slice + 16 * b + 4 * grp + v] = acc[rt][b][v];
            }
        }
    }
    if (RT == 1 && wave == 0 && lane < 16) {
        rec[16 + col] = -INFINITY;
        rec[JROWS + 16 + col] = 0.f;
    }
}

// exact rows per (sequence, query row): scores into LDS, max, sum, original-space value sum
template <bool F32>
__global__ __launch_bounds__(256) void jx_kernel(JDec p) {
    typedef typename std::conditional<F32, float, uint16_t>::type ET;
    __shared__ float xs[JX_CAP];
    __shared__ float red[256];
    const int s = blockIdx.x / p.rows, row = blockIdx.x % p.rows;
    const JSeq& S = p.seq[s];
    const int h = row % p.H, query = row / p.H, g = h / p.hpg;
    const ET* q = reinterpret_cast<const ET*>(S.q) + ((int64_t)query * p.H + h) * D;
    const ET* kx = reinterpret_cast<const ET*>(S.kx) + (int64_t)g * p.cap * D;
    const ET* vx = reinterpret_cast<const ET*>(S.vx) + (int64_t)g * p.cap * D;
    const int ne = (int)S.n_exact;
    const int tid = threadIdx.x;
    float mloc = -INFINITY;
    for (int e = tid; e < ne; e += 256) {
        float a = 0.f;
        for (int i = 0; i < D; ++i) a = fmaf(elem_f(q[i]), elem_f(kx[(int64_t)e * D + i]), a);
        a *= 0.08838834764831845f;
        xs[e] = a;
        mloc = fmaxf(mloc, a);
    }
    red[tid] = mloc;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (tid < o) red[tid] = fmaxf(red[tid], red[tid + o]);
        __syncthreads();
    }
    const float M = red[0];
    __syncthreads();
    float lloc = 0.f;
    for (int e = tid; e < ne; e += 256) {
        const float pe = fast_exp(xs[e] - M);
        xs[e] = pe;
        lloc += pe;
    }
    red[tid] = lloc;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (tid < o) red[tid] += red[tid + o];
        __syncthreads();
    }
    float* xr = p.xrec + ((int64_t)s * JROWS + row) * (2 + D);
    if (tid < D) {
        float a = 0.f;
        for (int e = 0; e < ne; ++e) a = fmaf(xs[e], elem_f(vx[(int64_t)e * D + tid]), a);
        xr[2 + tid] = a;
    }
    if (tid == 0) { xr[0] = M; xr[1] = red[0]; }
}

// combined rank-space sums per (sequence, row, 64 coefficients): the records' factors
// exp(m_x - M) once per workgroup, then 4 groups of threads over the records (fixed order
// within a group, then the 4 groups in order); workgroup 0 of a row records (M, L)
constexpr int JM_MAXWG = 256;      // records per sequence at most (joint_plan)
__global__ __launch_bounds__(256) void jm1_kernel(JDec p) {
    __shared__ float fx[JM_MAXWG];
    __shared__ float red[256];
    const int kb_n = p.R / 64;
    const int s = blockIdx.x / (p.rows * kb_n), rem = blockIdx.x % (p.rows * kb_n);
    const int row = rem / kb_n, kb = rem % kb_n;
    const int tid = threadIdx.x;
    const int64_t rs = JREC_HEAD + (int64_t)JROWS * p.R;
    const float* rec = p.rec + (int64_t)s * p.n_wg * rs;
    const float* xr = p.xrec + ((int64_t)s * JROWS + row) * (2 + D);
    const float mx = tid < p.n_wg ? rec[tid * rs + row] : -INFINITY;
    const float lx = tid < p.n_wg ? rec[tid * rs + JROWS + row] : 0.f;
    red[tid] = mx;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (tid < o) red[tid] = fmaxf(red[tid], red[tid + o]);
        __syncthreads();
    }
    const float M = fmaxf(red[0], xr[0]);
    __syncthreads();
    const float f = mx == -INFINITY ? 0.f : fast_exp(mx - M);
    if (tid < p.n_wg) fx[tid] = f;
    red[tid] = f * lx;
    __syncthreads();
    for (int o = 128; o > 0; o >>= 1) {
        if (tid < o) red[tid] += red[tid + o];
        __syncthreads();
    }
    if (kb == 0 && tid == 0) {
        p.ml[((int64_t)s * JROWS + row) * 2] = M;
        p.ml[((int64_t)s * JROWS + row) * 2 + 1] = red[0] + xr[1] * fast_exp(xr[0] - M);
    }
    __syncthreads();
    const int kk = tid & 63, xg = tid >> 6;
    const float* src = rec + JREC_HEAD + (int64_t)row * p.R + kb * 64 + kk;
    float a = 0.f;
#pragma unroll 8
    for (int x = xg; x < p.n_wg; x += 4) a = fmaf(fx[x], src[x * rs], a);
    red[tid] = a;
    __syncthreads();
    if (tid < 64)
        p.comb[((int64_t)s * JROWS + row) * p.R + kb * 64 + tid] = ((red[tid] + red[tid + 64]) + red[tid + 128]) + red[tid + 192];
}

// out = (W_V,g^T comb + exp(m_x - M) acc_x) / L for every query row of KV head g: a workgroup
// per (sequence, g, 32 output coordinates), 8 groups of 32 threads over the coefficients (the
// basis entry read once for all of g's rows), the 8 partial sums added in order
constexpr int JM2_ROWS = JROWS;
constexpr int JM2_KC = 256;        // coefficients per workgroup
constexpr int JM2_NP = 8;          // partial sums per chunk (thread groups)
__global__ __launch_bounds__(256) void jm2_kernel_part(JDec p, float* part) {
    __shared__ float cbs[JM2_ROWS][JM2_KC];
    __shared__ int rowof[JM2_ROWS];
    const int nkc = p.R / JM2_KC;
    const int s = blockIdx.x / (p.G * 4 * nkc);
    int rem = blockIdx.x % (p.G * 4 * nkc);
    const int g = rem / (4 * nkc);
    rem %= 4 * nkc;
    const int ib = rem / nkc, kc = rem % nkc;
    const int tid = threadIdx.x, i = ib * 32 + (tid & 31), kg = tid >> 5;
    const int Dz = 2 * p.G * D;
    const int k0 = kc * JM2_KC;
    const int nr = (p.rows / p.H) * p.hpg;      // head g's rows: query * H + g hpg + hh
    // this thread's basis entries W[k0 + kg + 8 m][(G + g) d + i], all loads in flight
    const float* w = p.W + (int64_t)(k0 + kg) * Dz + (p.G + g) * D + i;
    float wv[JM2_KC / JM2_NP];
#pragma unroll
    for (int m = 0; m < JM2_KC / JM2_NP; ++m) wv[m] = w[(int64_t)(JM2_NP * m) * Dz];
    if (tid < JM2_ROWS) rowof[tid] = tid < nr ? (tid / p.hpg) * p.H + g * p.hpg + tid % p.hpg : 0;
    __syncthreads();
    const float* comb = p.comb + (int64_t)s * JROWS * p.R + k0;
    for (int e = tid; e < nr * JM2_KC; e += 256) {
        const int r = e / JM2_KC, kk = e % JM2_KC;
        cbs[r][kk] = comb[(int64_t)rowof[r] * p.R + kk];
    }
    __syncthreads();
    float* dst = part + ((((int64_t)s * p.G + g) * (JM2_NP * nkc) + kc * JM2_NP + kg) * JM2_ROWS) * D + i;
    for (int r = 0; r < nr; ++r) {
        float a = 0.f;
#pragma unroll
        for (int m = 0; m < JM2_KC / JM2_NP; ++m) a = fmaf(wv[m], cbs[r][kg + JM2_NP * m], a);
        dst[r * D] = a;
    }
}

template <bool F32>
__global__ __launch_bounds__(D) void jm2_kernel(JDec p, const float* part) {
    typedef typename std::conditional<F32, float, uint16_t>::type ET;
    const int s = blockIdx.x / p.rows, row = blockIdx.x % p.rows;
    const int h = row % p.H, query = row / p.H, g = h / p.hpg;
    const int r = query * p.hpg + h % p.hpg;      // the row's index among head g's rows
    const int i = threadIdx.x;
    const int np = JM2_NP * (p.R / JM2_KC);
    const float* src = part + ((((int64_t)s * p.G + g) * np) * JM2_ROWS + r) * D + i;
    float a = 0.f;
#pragma unroll 8
    for (int x = 0; x < np; ++x) a += src[(int64_t)x * JM2_ROWS * D];
    const float M = p.ml[((int64_t)s * JROWS + row) * 2], L = p.ml[((int64_t)s * JROWS + row) * 2 + 1];
    const float* xr = p.xrec + ((int64_t)s * JROWS + row) * (2 + D);
    a = (a + fast_exp(xr[0] - M) * xr[2 + i]) / L;
    ET* out = reinterpret_cast<ET*>(p.seq[s].out) + ((int64_t)query * p.H + h) * D;
    out[i] = to_elem<ET>(a);
}

// the window rows stay exact: dst[g][e] = src[N + e][g] for K and V, 16 bytes per thread
__global__ __launch_bounds__(256) void jwin_kernel(const uint8_t* __restrict__ K, const uint8_t* __restrict__ V,
                                                   uint8_t* __restrict__ kx, uint8_t* __restrict__ vx, int64_t N,
                                                   int G, int w, int64_t cap, int row_bytes) {
    const int upr = row_bytes / 16;
    const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t total = 2 * (int64_t)w * G * upr;
    if (gid >= total) return;
    const int kv = (int)(gid / ((int64_t)w * G * upr));
    const int64_t r = gid % ((int64_t)w * G * upr);
    const int e = (int)(r / (G * upr)), g = (int)((r / upr) % G), u = (int)(r % upr);
    const uint8_t* src = (kv ? V : K) + ((N + e) * G + g) * (int64_t)row_bytes + 16 * u;
    uint8_t* dst = (kv ? vx : kx) + ((int64_t)g * cap + e) * row_bytes + 16 * u;
    *reinterpret_cast<u32x4*>(dst) = *reinterpret_cast<const u32x4*>(src);
}

hipError_t launch_joint_window(const varrate_shape& sh, const void* K, const void* V, varrate_jcache& c,
                               hipStream_t st) {
    const int row_bytes = D * (sh.dtype == VARRATE_BF16 ? 2 : 4);
    const int64_t total = 2 * (int64_t)sh.w * sh.G * (row_bytes / 16);
    jwin_kernel<<<(unsigned)((total + 255) / 256), 256, 0, st>>>((const uint8_t*)K, (const uint8_t*)V,
                                                                 (uint8_t*)c.k_exact, (uint8_t*)c.v_exact,
                                                                 sh.n - sh.w, sh.G, sh.w, c.cap, row_bytes);
    return hipGetLastError();
}

struct JPlan { int n_wg, tpw, total_tiles; };

static JPlan joint_plan(const varrate_shape& sh, int S) {
    JPlan pl;
    const int64_t N = sh.n - sh.w;
    pl.total_tiles = (int)((N + 15) / 16);
    const int ns = S < JSEQ ? S : JSEQ;
    int want = 256 / ns;                        // about one workgroup per CU per launch
    want = want < 1 ? 1 : (want > JM_MAXWG ? JM_MAXWG : want);
    pl.tpw = (pl.total_tiles + want - 1) / want;
    pl.n_wg = (pl.total_tiles + pl.tpw - 1) / pl.tpw;
    return pl;
}

size_t joint_decode_ws_bytes(const varrate_shape& sh, int R, int S, int Q) {
    (void)Q;
    const JPlan pl = joint_plan(sh, S);
    const size_t ns = (size_t)S;
    return align256(ns * JROWS * R * 4) + align256(ns * pl.n_wg * (JREC_HEAD + (size_t)JROWS * R) * 4) +
           align256(ns * JROWS * (2 + D) * 4) + align256(ns * JROWS * R * 4) + align256(ns * JROWS * 2 * 4) +
           align256(ns * sh.G * (JM2_NP * (size_t)R / JM2_KC) * JM2_ROWS * D * 4);
}

hipError_t launch_joint_decode(const varrate_shape& sh, int R, const varrate_jcache* caches, int S, const void* q,
                               int Q, const float* W, void* out, uint8_t* ws, hipStream_t st) {
    const JPlan pl = joint_plan(sh, S);
    const int rows = Q * sh.H;
    if (rows > JROWS) return hipErrorInvalidValue;
    const size_t es = sh.dtype == VARRATE_BF16 ? 2 : 4;
    const size_t qstride = (size_t)Q * sh.H * D * es;
    const size_t ns_all = (size_t)S;
    uint8_t* b = ws;
    float* qp = (float*)b;   b += align256(ns_all * JROWS * R * 4);
    float* rec = (float*)b;  b += align256(ns_all * pl.n_wg * (JREC_HEAD + (size_t)JROWS * R) * 4);
    float* xrec = (float*)b; b += align256(ns_all * JROWS * (2 + D) * 4);
    float* comb = (float*)b; b += align256(ns_all * JROWS * R * 4);
    float* ml = (float*)b;   b += align256(ns_all * JROWS * 2 * 4);
    float* part = (float*)b;
    const bool f32 = sh.dtype != VARRATE_BF16;
    for (int s0 = 0; s0 < S; s0 += JSEQ) {
        const int ns = S - s0 < JSEQ ? S - s0 : JSEQ;
        JDec p;
        for (int i = 0; i < JSEQ; ++i) {
            const varrate_jcache& c = caches[s0 + (i < ns ? i : 0)];
            const int si = s0 + (i < ns ? i : 0);
            p.seq[i] = JSeq{c.coef, c.rank, c.offset, c.k_exact, c.v_exact, (const uint8_t*)q + si * qstride,
                            (uint8_t*)out + si * qstride, c.n_exact};
        }
        p.W = W;
        p.qp = qp + (size_t)s0 * JROWS * R;
        p.rec = rec + (size_t)s0 * pl.n_wg * (JREC_HEAD + (size_t)JROWS * R);
        p.xrec = xrec + (size_t)s0 * JROWS * (2 + D);
        p.comb = comb + (size_t)s0 * JROWS * R;
        p.ml = ml + (size_t)s0 * JROWS * 2;
        p.N = sh.n - sh.w;
        p.cap = caches[s0].cap;
        p.G = sh.G;
        p.H = sh.H;
        p.hpg = sh.H / sh.G;
        p.rows = rows;
        p.R = R;
        p.n_wg = pl.n_wg;
        p.tpw = pl.tpw;
        p.total_tiles = pl.total_tiles;
        const unsigned nq = (unsigned)(ns * JROWS * (R / 64));
        const unsigned nd = (unsigned)(ns * pl.n_wg);
        const unsigned nx = (unsigned)(ns * rows);
        const unsigned n1 = (unsigned)(ns * rows * (R / 64));
        const unsigned n2 = (unsigned)(ns * sh.G * 4 * (R / JM2_KC));
        float* pt = part + (size_t)s0 * sh.G * (JM2_NP * (size_t)R / JM2_KC) * JM2_ROWS * D;
        if (f32) {
            jq_kernel<true><<<nq, 256, 0, st>>>(p);
            if (rows > 16) jd_kernel<true, 2><<<nd, JD_T, 0, st>>>(p);
            else jd_kernel<true, 1><<<nd, JD_T, 0, st>>>(p);
            jx_kernel<true><<<nx, 256, 0, st>>>(p);
            jm1_kernel<<<n1, 256, 0, st>>>(p);
            jm2_kernel_part<<<n2, 256, 0, st>>>(p, pt);
            jm2_kernel<true><<<nx, D, 0, st>>>(p, pt);
        } else {
            jq_kernel<false><<<nq, 256, 0, st>>>(p);
            if (rows > 16) jd_kernel<false, 2><<<nd, JD_T, 0, st>>>(p);
            else jd_kernel<false, 1><<<nd, JD_T, 0, st>>>(p);
            jx_kernel<false><<<nx, 256, 0, st>>>(p);
            jm1_kernel<<<n1, 256, 0, st>>>(p);
            jm2_kernel_part<<<n2, 256, 0, st>>>(p, pt);
            jm2_kernel<false><<<nx, D, 0, st>>>(p, pt);
        }
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace vr
