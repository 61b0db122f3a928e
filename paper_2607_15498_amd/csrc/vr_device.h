// Device helpers shared by the CDNA4 (gfx950) kernels of the variable-rank codec.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vr {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int D = 128;          // head dim = basis rank R
constexpr int WAVE = 64;

// ---- bf16 <-> fp32 -------------------------------------------------------------------
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// element <-> fp32 for the storage types (bf16 bits in uint16_t, or fp32)
__device__ __forceinline__ float elem_f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ __forceinline__ float elem_f(float x) { return x; }

// fp32 -> bf16 bits, round to nearest even (inputs are finite).
__device__ __forceinline__ uint32_t f32_to_bf16(float x) {
    uint32_t u = __float_as_uint(x);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
template <typename ET> __device__ __forceinline__ ET to_elem(float x);
template <> __device__ __forceinline__ uint16_t to_elem<uint16_t>(float x) { return (uint16_t)f32_to_bf16(x); }
template <> __device__ __forceinline__ float to_elem<float>(float x) { return x; }

// x = hi + lo to about 2^-17 relative: hi = bf16(x), lo = bf16(x - hi).
__device__ __forceinline__ void split_bf16(float x, uint32_t& hi, uint32_t& lo) {
    hi = f32_to_bf16(x);
    lo = f32_to_bf16(x - __uint_as_float(hi << 16));
}
__device__ __forceinline__ uint32_t pack2(uint32_t lo16, uint32_t hi16) { return lo16 | (hi16 << 16); }

// Two fp32 -> packed bf16x2 (a in the low half), round to nearest even, by the gfx950
// conversion instruction.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t cvt_bf16x2(float a, float b) {
    const bf16x2_t v = {(__bf16)a, (__bf16)b};
    return __builtin_bit_cast(uint32_t, v);
}
// (hi, lo) bf16x2 pairs of two fp32 values.
__device__ __forceinline__ void split2(float a, float b, uint32_t& hi, uint32_t& lo) {
    hi = cvt_bf16x2(a, b);
    lo = cvt_bf16x2(a - bf_lo(hi), b - bf_hi(hi));
}

// 8 fp32 -> (hi, lo) bf16x8 fragments.
__device__ __forceinline__ void split8(const float* x, u32x4& hi, u32x4& lo) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        uint32_t h, l;
        split2(x[2 * k], x[2 * k + 1], h, l);
        hi[k] = h;
        lo[k] = l;
    }
}

// ---- MFMA -------------------------------------------------------------------------------
// D(16x16 fp32) += A(16x32 bf16) * B(32x16 bf16).  Operand lane layout (wave64):
//   A: lane l holds row (l % 16), 8 K-elements of group (l / 16);
//   B: lane l holds column (l % 16), the same 8 K-elements of group (l / 16);
//   C: lane l holds column (l % 16), rows 4 (l / 16) + v, v = 0..3.
// A and B share the K-element assignment, so any fixed mapping of (group, element) to the
// contraction index gives the same product.
__device__ __forceinline__ f32x4 mfma(const u32x4& a, const u32x4& b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// ---- loads ---------------------------------------------------------------------------
// 16 bytes from a 2-byte aligned address (gfx950 serves it with one dwordx4 load).
__device__ __forceinline__ u32x4 load16_a2(const uint16_t* p) {
    u32x4 v;
    __builtin_memcpy(&v, p, 16);
    return v;
}
__device__ __forceinline__ u32x4 load16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }

// Keep the first nv (0..8) bf16 elements of an 8-element fragment, zero the rest.
__device__ __forceinline__ u32x4 keep_first(u32x4 v, int nv) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        uint32_t m = nv >= 2 * k + 2 ? 0xFFFFFFFFu : (nv == 2 * k + 1 ? 0x0000FFFFu : 0u);
        v[k] &= m;
    }
    return v;
}

// ---- wave / block reductions ---------------------------------------------------------
__device__ __forceinline__ float shfl_xor_f(float v, int m) { return __shfl_xor(v, m, WAVE); }

__device__ __forceinline__ float wave_max16(float v) {   // over lanes sharing l/16 ... l%16
    v = fmaxf(v, shfl_xor_f(v, 1));
    v = fmaxf(v, shfl_xor_f(v, 2));
    v = fmaxf(v, shfl_xor_f(v, 4));
    v = fmaxf(v, shfl_xor_f(v, 8));
    return v;
}

// Reductions over the lane pairs (l, l ^ 16) and (l, l ^ 32) by the gfx950 permlane swaps
// (ALU ops, no LDS path, no lane-index arithmetic).  Both lanes of a pair receive the two
// values in the same order, so both compute bit-identical results.
__device__ __forceinline__ float xmax16(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xmax32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xsum16(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xsum32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Rotary embedding angle (Sec. 3.1 "Joint per-token vector"): cos and sin of p * theta for
// an integer position p < 2^24, with theta / (2 pi) given as the double-float fhi + flo.  The
// product's whole turns are removed exactly (fmaf returns p * fhi - prod exactly), and the
// remaining fraction of a turn (|r| < 1, error ~2^-25 turns) goes to the hardware sine and
// cosine, which take their argument in turns.
__device__ __forceinline__ void rope_cs(float p, float fhi, float flo, float& c, float& s) {
    const float prod = p * fhi;
    const float err = fmaf(p, fhi, -prod);
    const float r = (prod - rintf(prod)) + (err + p * flo);
    s = __builtin_amdgcn_sinf(r);
    c = __builtin_amdgcn_cosf(r);
}

// exp(x) on the hardware exp2 path (x * log2 e); -inf -> 0.
__device__ __forceinline__ float fast_exp(float x) { return __builtin_amdgcn_exp2f(x * 1.4426950408889634f); }

// Salience pooling terms (Sec. 3.2, after Eq. (4)): s_k = (sum over the G heads of the
// per-head column sums, fp32 in head order) / (w H), carried in fp64; the pooled value of a
// token is the centred 5-term sum of s in fixed order, divided by 5 and rounded to fp32.
// Used by the pooling kernel and by the compress path's fused pooling + range pass, so both
// produce the same bits.
constexpr int POOL_MAXG = 16;      // heads whose loads issue together
// the first POOL_MAXG heads' column sums of token k (0 <= k < N), loaded by the caller; the
// loads are unconditional (heads past G read head 0, and the sum skips them) so that they all
// issue before the first wait
__device__ __forceinline__ void pool_load(const float* __restrict__ s_part, int64_t N, int G, int64_t k,
                                          float (&part)[POOL_MAXG]) {
#pragma unroll
    for (int gg = 0; gg < POOL_MAXG; ++gg) part[gg] = s_part[(int64_t)(gg < G ? gg : 0) * N + k];
}
__device__ __forceinline__ double pool_sum(const float (&part)[POOL_MAXG], const float* __restrict__ s_part,
                                           int64_t N, int G, float inv_wh, int64_t k) {
    float s = 0.f;
#pragma unroll
    for (int gg = 0; gg < POOL_MAXG; ++gg)
        if (gg < G) s += part[gg];
    for (int gg = POOL_MAXG; gg < G; ++gg) s += s_part[(int64_t)gg * N + k];
    return (double)(s * inv_wh);
}
__device__ __forceinline__ double pool_term(const float* __restrict__ s_part, int64_t N, int G,
                                            float inv_wh, int64_t k) {
    if (k < 0 || k >= N) return 0.0;
    float part[POOL_MAXG];
    pool_load(s_part, N, G, k, part);
    return pool_sum(part, s_part, N, G, inv_wh, k);
}
// sv[i - 2 .. i + 2] are the terms around the token
__device__ __forceinline__ float pool5(const double* sv, int i) {
    const double acc = (((sv[i - 2] + sv[i - 1]) + sv[i]) + sv[i + 1]) + sv[i + 2];
    return (float)(acc / 5.0);
}

}  // namespace vr
