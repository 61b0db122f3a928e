// Rotary keys (Sec. 3.1 "Joint per-token vector"; Algorithm 1, first and last steps), gfx950.
//
// The caller's keys are post-RoPE in the rotate-half layout: coordinates i and i + 64 form
// pair i, turned at position p by p * theta_i.  The codec codes pre-RoPE keys, so compress
// un-rotates the coded tokens (position t for prompt token t) into a workspace copy held in
// the storage type and projects that; the window rows are copied unchanged (they stay exact
// and post-RoPE).  Decode rebuilds each coded key from its coefficients by MFMA against the
// key basis and rotates it back to its position; the kernels here prepare, once per call,
// the basis in MFMA fragment order (bf16 hi + lo parts) and the frequency table.
#include <cmath>

#include "vr_internal.h"

namespace vr {

RopeFreq rope_freq(const varrate_shape& sh) {
    RopeFreq f;
    const double inv2pi = 0.15915494309189533576888;   // 1 / (2 pi)
    for (int i = 0; i < D / 2; ++i) {
        const double t = (double)sh.rope_theta[i] * inv2pi;
        f.hi[i] = (float)t;
        f.lo[i] = (float)(t - (double)f.hi[i]);
    }
    return f;
}

// One thread per (token, head, 4 pairs): rows t < N are turned back by -t and rounded to the
// storage type, rows t >= N (the window) are copied.
template <typename ET>
__global__ __launch_bounds__(256) void rope_unrotate_kernel(const ET* __restrict__ K, ET* __restrict__ Kr,
                                                            int64_t n, int64_t N, int G, RopeFreq f) {
    __shared__ float fh_s[D / 2], fl_s[D / 2];
    if (threadIdx.x < D / 2) {
        // the argument table read at uniform indices only
        float h = 0.f, l = 0.f;
#pragma unroll
        for (int j = 0; j < D / 2; ++j)
            if ((int)threadIdx.x == j) { h = f.hi[j]; l = f.lo[j]; }
        fh_s[threadIdx.x] = h;
        fl_s[threadIdx.x] = l;
    }
    __syncthreads();
    const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t row = gid >> 4;                  // token * G + head
    const int i0 = 4 * (int)(gid & 15);            // first pair of the thread
    if (row >= n * G) return;
    const int64_t t = row / G;
    const ET* src = K + row * D;
    ET* dst = Kr + row * D;
    float x0[4], x1[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        x0[k] = elem_f(src[i0 + k]);
        x1[k] = elem_f(src[i0 + k + D / 2]);
    }
    if (t < N) {
        const float p = (float)t;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            float c, s;
            rope_cs(p, fh_s[i0 + k], fl_s[i0 + k], c, s);
            // rotation by -p: (x0 c + x1 s, x1 c - x0 s)
            const float a = x0[k] * c + x1[k] * s;
            const float b = x1[k] * c - x0[k] * s;
            x0[k] = a;
            x1[k] = b;
        }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        dst[i0 + k] = to_elem<ET>(x0[k]);
        dst[i0 + k + D / 2] = to_elem<ET>(x1[k]);
    }
}

hipError_t launch_rope_unrotate(const varrate_shape& sh, const void* K, void* Kr, hipStream_t st) {
    const RopeFreq f = rope_freq(sh);
    const int64_t N = sh.n - sh.w;
    const int64_t threads = sh.n * sh.G * 16;
    const unsigned blocks = (unsigned)((threads + 255) / 256);
    if (sh.dtype == VARRATE_BF16)
        rope_unrotate_kernel<uint16_t><<<blocks, 256, 0, st>>>((const uint16_t*)K, (uint16_t*)Kr, sh.n, N, sh.G, f);
    else
        rope_unrotate_kernel<float><<<blocks, 256, 0, st>>>((const float*)K, (float*)Kr, sh.n, N, sh.G, f);
    return hipGetLastError();
}

// Decode operands.  frags[g][s][b][part][lane] (u32x4): the A operand of the reconstruction
// MFMA K^T[dim][token] = sum_j P_K[j][dim] c[token][j] for dims 16 b .. 16 b + 15 and
// coefficients 32 s .. 32 s + 31: lane -> dim 16 b + (lane & 15), coefficients
// 32 s + 8 (lane >> 4) + 0..7, as bf16 hi (part 0) and lo (part 1) of the fp32 basis.
// freq[2 i], freq[2 i + 1]: the double-float theta_i / (2 pi).
__global__ __launch_bounds__(256) void rope_prep_kernel(const float* __restrict__ PK, u32x4* __restrict__ frags,
                                                        float* __restrict__ freq, int G, RopeFreq f) {
    const int gid = blockIdx.x * 256 + threadIdx.x;   // (g, s, b, lane)
    if (gid < 2 * (D / 2) && blockIdx.x == 0) {
        float v = 0.f;
#pragma unroll
        for (int j = 0; j < D / 2; ++j) {
            if (gid == 2 * j) v = f.hi[j];
            if (gid == 2 * j + 1) v = f.lo[j];
        }
        freq[gid] = v;
    }
    if (gid >= G * 4 * 8 * 64) return;
    const int lane = gid & 63, b = (gid >> 6) & 7, s = (gid >> 9) & 3, g = gid >> 11;
    const int dim = 16 * b + (lane & 15);
    const int j0 = 32 * s + 8 * (lane >> 4);
    const float* P = PK + (int64_t)g * D * D;
    float x[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = P[(j0 + e) * D + dim];
    u32x4 hi, lo;
    split8(x, hi, lo);
    u32x4* out = frags + ((((int64_t)g * 4 + s) * 8 + b) * 2) * 64;
    out[lane] = hi;
    out[64 + lane] = lo;
}

hipError_t launch_rope_prep(const varrate_shape& sh, const float* PK, void* frags, float* freq, hipStream_t st) {
    const RopeFreq f = rope_freq(sh);
    const int threads = sh.G * 4 * 8 * 64;
    rope_prep_kernel<<<(unsigned)((threads + 255) / 256), 256, 0, st>>>(PK, (u32x4*)frags, freq, sh.G, f);
    return hipGetLastError();
}

}  // namespace vr
