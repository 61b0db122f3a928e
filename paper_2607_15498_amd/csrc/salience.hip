// Observation-window salience (Sec. 3.2 Eq. (4)) and SnapKV pooling, gfx950.
//
// For KV head g the window queries of its H/G query heads form `rows` = (H/G) * w query
// rows (row rho = hh * w + i: query head g*(H/G)+hh, window query i at position n-w+i).
// Logits x = <q_rho, k_t> / sqrt(d) come from bf16 MFMA tiles (16 rows x 16 keys x 32 d);
// fp32 inputs are split into bf16 hi + lo parts (three products), keeping ~2^-16 accuracy.
//
//   pass 1 (sal_rowstats): per (row, key block) online max / sum of exp over the causal
//            range, from key tiles staged through LDS;
//   merge  (sal_merge):    per row, the global max M and 1/L;
//   pass 2 (sal_colsum):   per coded key t, sum over rows of exp(x - M) / L (every window
//            query sees every coded key, so no mask), summed over the group's rows in a
//            fixed order -> s_part[g][t];
//   pool   (sal_pool):     s_t = sum_g s_part[g][t] / (w H) (fixed order), then the centred
//            length-5 moving average with zero padding, rounded to fp32.
#include "vr_internal.h"

namespace vr {

constexpr int SAL_THREADS = 256;           // 4 waves
constexpr int SAL_KSUB = 64;               // keys staged in LDS at a time
constexpr int SAL_KB1 = 512;               // keys per pass-1 workgroup
constexpr int SAL_KB2 = 256;               // keys per pass-2 workgroup
constexpr int SAL_MAX_RT = 4;              // row tiles per wave (rows <= 4 * 16 * 4 = 256)

template <bool F32> struct KTile;
// bf16 keys: row of 128 bf16 = 256 B, padded to 272 B to spread LDS banks.
template <> struct KTile<false> {
    static constexpr int ROW_U32 = 68;
};
// fp32 keys are staged as split hi/lo bf16 rows (2 x 272 B).
template <> struct KTile<true> {
    static constexpr int ROW_U32 = 136;
};

// Keys of one staging step: SAL_KSUB keys x 16 pieces of 8 elements; each thread holds
// 4 pieces (bf16: 16 bytes each; fp32: 32 bytes each, split into hi/lo when stored).
template <bool F32> struct KRegs { u32x4 a[4]; u32x4 b[4]; };

template <bool F32>
__device__ __forceinline__ void load_keys(KRegs<F32>& r, const void* K, int64_t n, int G, int g, int64_t k0) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int idx = threadIdx.x + k * SAL_THREADS;
        const int key = idx >> 4, ch = idx & 15;
        const int64_t t = k0 + key;
        r.a[k] = r.b[k] = u32x4{0, 0, 0, 0};
        if (t < n) {
            if constexpr (!F32) {
                r.a[k] = load16((const uint16_t*)K + ((t * G + g) * D + ch * 8));
            } else {
                const float* src = (const float*)K + ((t * G + g) * D + ch * 8);
                r.a[k] = load16(src);
                r.b[k] = load16(src + 4);
            }
        }
    }
}

template <bool F32>
__device__ __forceinline__ void store_keys(uint32_t* lds, const KRegs<F32>& r) {
    constexpr int RU = KTile<F32>::ROW_U32;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int idx = threadIdx.x + k * SAL_THREADS;
        const int key = idx >> 4, ch = idx & 15;
        if constexpr (!F32) {
            *reinterpret_cast<u32x4*>(lds + key * RU + ch * 4) = r.a[k];
        } else {
            float x[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) { x[e] = __uint_as_float(r.a[k][e]); x[4 + e] = __uint_as_float(r.b[k][e]); }
            u32x4 hi, lo;
            split8(x, hi, lo);
            *reinterpret_cast<u32x4*>(lds + key * RU + ch * 4) = hi;
            *reinterpret_cast<u32x4*>(lds + key * RU + 68 + ch * 4) = lo;
        }
    }
}

// Query fragments (A operand) for row tile rt: lane row = 16 rt + l%16, K group l/16.
template <bool F32>
__device__ __forceinline__ void load_qfrag(const void* Qw, int H, int w, int hpg, int g, int rows,
                                           int rt, u32x4 (&qh)[4], u32x4 (&ql)[4]) {
    const int lane = threadIdx.x & 63;
    const int rho = rt * 16 + (lane & 15);
    const int grp = lane >> 4;
    const bool ok = rho < rows;
    const int hh = ok ? rho / w : 0, i = ok ? rho % w : 0;
    const int64_t base = ((int64_t)i * H + (g * hpg + hh)) * D;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const int c0 = 32 * s + 8 * grp;
        if constexpr (!F32) {
            qh[s] = ok ? load16((const uint16_t*)Qw + base + c0) : u32x4{0, 0, 0, 0};
            ql[s] = u32x4{0, 0, 0, 0};
        } else {
            float x[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            if (ok) {
                const float* src = (const float*)Qw + base + c0;
                u32x4 a = load16(src), b = load16(src + 4);
                for (int e = 0; e < 4; ++e) { x[e] = __uint_as_float(a[e]); x[4 + e] = __uint_as_float(b[e]); }
            }
            split8(x, qh[s], ql[s]);
        }
    }
}

// Logit tile: rows 16 rt.., keys kt*16.. of the staged block (C layout: lane col = key).
template <bool F32>
__device__ __forceinline__ f32x4 logit_tile(const uint32_t* lds, int kt, const u32x4 (&qh)[4],
                                            const u32x4 (&ql)[4]) {
    constexpr int RU = KTile<F32>::ROW_U32;
    const int lane = threadIdx.x & 63;
    const uint32_t* row = lds + (kt * 16 + (lane & 15)) * RU + (lane >> 4) * 4;
    f32x4 c = {0, 0, 0, 0};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        u32x4 kh = *reinterpret_cast<const u32x4*>(row + s * 16);
        c = mfma(qh[s], kh, c);
        if constexpr (F32) {
            u32x4 kl = *reinterpret_cast<const u32x4*>(row + 68 + s * 16);
            c = mfma(ql[s], kh, c);
            c = mfma(qh[s], kl, c);
        }
    }
    return c;
}

// ----------------------------------------------------------------------------------------
// pass 1: stats[(g * rows + rho) * nkb + kb] = (max, sum exp(x - max)) over this block's
// causal keys.  Grid (nkb, G).
template <bool F32>
__global__ __launch_bounds__(SAL_THREADS) void sal_rowstats(const void* __restrict__ K,
                                                            const void* __restrict__ Qw,
                                                            int64_t n, int G, int H, int w,
                                                            float2* __restrict__ stats, int nkb) {
    __shared__ __attribute__((aligned(16))) uint32_t lds[SAL_KSUB * KTile<F32>::ROW_U32];
    const int kb = blockIdx.x, g = blockIdx.y;
    const int hpg = H / G, rows = hpg * w, nrt = (rows + 15) / 16;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int64_t kbeg = (int64_t)kb * SAL_KB1;
    const int64_t kend = kbeg + SAL_KB1 < n ? kbeg + SAL_KB1 : n;

    u32x4 qh[SAL_MAX_RT][4], ql[SAL_MAX_RT][4];
    float m[SAL_MAX_RT][4], l[SAL_MAX_RT][4];
#pragma unroll
    for (int j = 0; j < SAL_MAX_RT; ++j) {
        const int rt = wave + 4 * j;
        if (rt < nrt) load_qfrag<F32>(Qw, H, w, hpg, g, rows, rt, qh[j], ql[j]);
#pragma unroll
        for (int v = 0; v < 4; ++v) { m[j][v] = -INFINITY; l[j][v] = 0.f; }
    }
    const float scale = 0.08838834764831845f;  // 1/sqrt(128)

    KRegs<F32> kr;
    load_keys<F32>(kr, K, n, G, g, kbeg);
    for (int64_t k0 = kbeg; k0 < kend; k0 += SAL_KSUB) {
        __syncthreads();
        store_keys<F32>(lds, kr);
        __syncthreads();
        if (k0 + SAL_KSUB < kend) load_keys<F32>(kr, K, n, G, g, k0 + SAL_KSUB);
#pragma unroll
        for (int j = 0; j < SAL_MAX_RT; ++j) {
            const int rt = wave + 4 * j;
            if (rt >= nrt) continue;
            for (int kt = 0; kt < SAL_KSUB / 16; ++kt) {
                const int64_t t = k0 + kt * 16 + (lane & 15);
                if (k0 + kt * 16 >= kend) break;
                f32x4 c = logit_tile<F32>(lds, kt, qh[j], ql[j]);
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int rho = rt * 16 + (lane >> 4) * 4 + v;
                    const int i = rho % w;
                    const bool vis = rho < rows && t < kend && t <= n - w + i;
                    const float x = c[v] * scale;
                    if (vis) {
                        // online max/sum; rescale only when the max moves up
                        if (x > m[j][v]) {
                            l[j][v] = l[j][v] * fast_exp(m[j][v] - x) + 1.f;
                            m[j][v] = x;
                        } else {
                            l[j][v] += fast_exp(x - m[j][v]);
                        }
                    }
                }
            }
        }
    }
    // combine the 16 lanes that share a row (lane bits 0..3)
#pragma unroll
    for (int j = 0; j < SAL_MAX_RT; ++j) {
        const int rt = wave + 4 * j;
        if (rt >= nrt) continue;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            float mm = m[j][v], ll = l[j][v];
#pragma unroll
            for (int off = 1; off < 16; off <<= 1) {
                const float mo = shfl_xor_f(mm, off), lo = shfl_xor_f(ll, off);
                const float mn = fmaxf(mm, mo);
                const float a = mm == -INFINITY ? 0.f : ll * fast_exp(mm - mn);
                const float b = mo == -INFINITY ? 0.f : lo * fast_exp(mo - mn);
                mm = mn;
                ll = a + b;
            }
            const int rho = rt * 16 + (lane >> 4) * 4 + v;
            if ((lane & 15) == 0 && rho < rows)
                stats[((int64_t)g * rows + rho) * nkb + kb] = make_float2(mm, ll);
        }
    }
}

// merge: ML[g * rows + rho] = (M, 1/L).  16 threads per row read its block partials in
// parallel and combine them with shuffles.
__global__ __launch_bounds__(256) void sal_merge(const float2* __restrict__ stats, int nkb,
                                                 int total_rows, float2* __restrict__ ML) {
    const int r = blockIdx.x * 16 + (threadIdx.x >> 4), k = threadIdx.x & 15;
    float m = -INFINITY, l = 0.f;
    if (r < total_rows) {
        const float2* s = stats + (int64_t)r * nkb;
        for (int b = k; b < nkb; b += 16) {
            const float2 v = s[b];
            if (v.x == -INFINITY) continue;
            const float mn = fmaxf(m, v.x);
            l = (m == -INFINITY ? 0.f : l * fast_exp(m - mn)) + v.y * fast_exp(v.x - mn);
            m = mn;
        }
    }
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) {
        const float mo = shfl_xor_f(m, off), lo = shfl_xor_f(l, off);
        const float mn = fmaxf(m, mo);
        const float a = m == -INFINITY ? 0.f : l * fast_exp(m - mn);
        const float b = mo == -INFINITY ? 0.f : lo * fast_exp(mo - mn);
        m = mn;
        l = a + b;
    }
    if (k == 0 && r < total_rows) ML[r] = make_float2(m, 1.f / l);
}

// pass 2: s_part[g * N + t] = sum over the group's rows of exp(x - M) / L, t < N.
// Grid (ceil(N / SAL_KB2), G).
template <bool F32>
__global__ __launch_bounds__(SAL_THREADS) void sal_colsum(const void* __restrict__ K,
                                                          const void* __restrict__ Qw,
                                                          int64_t n, int G, int H, int w,
                                                          const float2* __restrict__ ML,
                                                          float* __restrict__ s_part) {
    __shared__ __attribute__((aligned(16))) uint32_t lds[SAL_KSUB * KTile<F32>::ROW_U32];
    __shared__ float colsum[4][SAL_KSUB];
    const int g = blockIdx.y;
    const int64_t N = n - w;
    const int hpg = H / G, rows = hpg * w, nrt = (rows + 15) / 16;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int64_t kbeg = (int64_t)blockIdx.x * SAL_KB2;
    const int64_t kend = kbeg + SAL_KB2 < N ? kbeg + SAL_KB2 : N;

    u32x4 qh[SAL_MAX_RT][4], ql[SAL_MAX_RT][4];
    float rm[SAL_MAX_RT][4], rinv[SAL_MAX_RT][4];
#pragma unroll
    for (int j = 0; j < SAL_MAX_RT; ++j) {
        const int rt = wave + 4 * j;
        if (rt < nrt) load_qfrag<F32>(Qw, H, w, hpg, g, rows, rt, qh[j], ql[j]);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int rho = rt * 16 + (lane >> 4) * 4 + v;
            float2 mlv = (rt < nrt && rho < rows) ? ML[(int64_t)g * rows + rho] : make_float2(INFINITY, 0.f);
            rm[j][v] = mlv.x;
            rinv[j][v] = mlv.y;
        }
    }
    const float scale = 0.08838834764831845f;

    KRegs<F32> kr;
    load_keys<F32>(kr, K, n, G, g, kbeg);
    for (int64_t k0 = kbeg; k0 < kend; k0 += SAL_KSUB) {
        __syncthreads();
        store_keys<F32>(lds, kr);
        __syncthreads();
        if (k0 + SAL_KSUB < kend) load_keys<F32>(kr, K, n, G, g, k0 + SAL_KSUB);
        for (int kt = 0; kt < SAL_KSUB / 16; ++kt) {
            float acc = 0.f;   // this lane's key column: sum over the wave's rows
#pragma unroll
            for (int j = 0; j < SAL_MAX_RT; ++j) {
                const int rt = wave + 4 * j;
                if (rt >= nrt) continue;
                f32x4 c = logit_tile<F32>(lds, kt, qh[j], ql[j]);
#pragma unroll
                for (int v = 0; v < 4; ++v) acc += fast_exp(c[v] * scale - rm[j][v]) * rinv[j][v];
            }
            acc += shfl_xor_f(acc, 16);
            acc += shfl_xor_f(acc, 32);
            if (lane < 16) colsum[wave][kt * 16 + lane] = acc;
        }
        __syncthreads();
        if (threadIdx.x < SAL_KSUB) {
            const int64_t t = k0 + threadIdx.x;
            if (t < kend) {
                const int kk = threadIdx.x;
                s_part[(int64_t)g * N + t] = ((colsum[0][kk] + colsum[1][kk]) + colsum[2][kk]) + colsum[3][kk];
            }
        }
    }
}

// pool: sbar[t] = (s_{t-2} + ... + s_{t+2}) / 5 with s_k = sum_g s_part[g][k] / (w H).
__global__ void sal_pool(const float* __restrict__ s_part, int64_t N, int G, float inv_wh,
                         float* __restrict__ sbar) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= N) return;
    double acc = 0.0;
    for (int64_t k = t - 2; k <= t + 2; ++k) {
        if (k < 0 || k >= N) continue;
        float s = 0.f;
        for (int g = 0; g < G; ++g) s += s_part[(int64_t)g * N + k];
        acc += (double)(s * inv_wh);
    }
    sbar[t] = (float)(acc / 5.0);
}

// ----------------------------------------------------------------------------------------
size_t salience_ws_bytes(const varrate_shape& sh) {
    const int rows = (sh.H / sh.G) * sh.w;
    const int64_t nkb = (sh.n + SAL_KB1 - 1) / SAL_KB1;
    const int64_t N = sh.n - sh.w;
    return align256((size_t)sh.G * rows * nkb * sizeof(float2)) +
           align256((size_t)sh.G * rows * sizeof(float2)) + align256((size_t)sh.G * N * sizeof(float));
}

hipError_t launch_salience(const varrate_shape& sh, const void* K, const void* Qw, float* sbar,
                           uint8_t* ws, hipStream_t st) {
    const int rows = (sh.H / sh.G) * sh.w;
    const int nkb = (int)((sh.n + SAL_KB1 - 1) / SAL_KB1);
    const int64_t N = sh.n - sh.w;
    float2* stats = (float2*)ws;
    ws += align256((size_t)sh.G * rows * nkb * sizeof(float2));
    float2* ML = (float2*)ws;
    ws += align256((size_t)sh.G * rows * sizeof(float2));
    float* s_part = (float*)ws;

    dim3 g1(nkb, sh.G), g2((unsigned)((N + SAL_KB2 - 1) / SAL_KB2), sh.G);
    const int tr = sh.G * rows;
    if (sh.dtype == VARRATE_BF16) {
        sal_rowstats<false><<<g1, SAL_THREADS, 0, st>>>(K, Qw, sh.n, sh.G, sh.H, sh.w, stats, nkb);
        sal_merge<<<(tr + 15) / 16, 256, 0, st>>>(stats, nkb, tr, ML);
        sal_colsum<false><<<g2, SAL_THREADS, 0, st>>>(K, Qw, sh.n, sh.G, sh.H, sh.w, ML, s_part);
    } else {
        sal_rowstats<true><<<g1, SAL_THREADS, 0, st>>>(K, Qw, sh.n, sh.G, sh.H, sh.w, stats, nkb);
        sal_merge<<<(tr + 15) / 16, 256, 0, st>>>(stats, nkb, tr, ML);
        sal_colsum<true><<<g2, SAL_THREADS, 0, st>>>(K, Qw, sh.n, sh.G, sh.H, sh.w, ML, s_part);
    }
    sal_pool<<<(unsigned)((N + 255) / 256), 256, 0, st>>>(s_part, N, sh.G,
                                                           1.0f / ((float)sh.w * (float)sh.H), sbar);
    return hipGetLastError();
}

}  // namespace vr
