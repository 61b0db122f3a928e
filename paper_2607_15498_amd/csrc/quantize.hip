// Group-wise b-bit quantisation of a compressed layer's coefficients (Sec. 3.3
// "Composability": the coefficients are quantised on their own, the allocation unchanged).
//
// Groups: one stored position's coefficients of one head and stream (K or V) in one
// 32-coordinate segment.  Symmetric absmax per group: with Qmax = 2^(b-1) - 1,
//     sc = binary16(fp32(amax / Qmax)),   k = clamp(rint(fp32(x / sc)), -Qmax, Qmax),
// correctly rounded fp32 divisions, ties to even; a group with sc = 0 codes 0.  The input x
// is the stored bf16 coefficient; entries past a position's rank are stored zeros, so they
// change neither amax nor their code (0).
//
// Output layout, per head stream, tile by tile in the same storage order as the coefficient
// layout (chunk c at qchunk_off[c] bytes): a tile of size m (its first position's rank)
// takes mq = m rounded up to a multiple of 8 coordinates and KS = ceil(m / 32) groups per
// position:
//   K stream: 16 rows of mq codes (code (i, j) at bit b (i mq + j)), then KS x 16 scales;
//   V stream: mq rows of 16 codes (code (j, i) at bit b (16 j + i)), then KS x 16 scales;
// codes are two's complement b-bit fields from bit 0 of the tile upward, scales binary16
// at [s][position].  Tile bytes: 2 mq b + 32 KS (a multiple of 16).
//
// Two launches: one workgroup sums the tile sizes of every chunk and scans them into
// qchunk_off; then a workgroup per (chunk, head, stream) writes that chunk's tiles.
#include "vr_internal.h"

namespace vr {

constexpr int QZ_SCAN_THREADS = 1024;

__host__ __device__ constexpr uint32_t qz_tile_bytes(uint32_t m, int b) {
    return m == 0 ? 0u : 2u * ((m + 7u) & ~7u) * (uint32_t)b + 32u * ((m + 31u) / 32u);
}

__global__ __launch_bounds__(QZ_SCAN_THREADS) void qz_scan_kernel(const uint8_t* __restrict__ srank,
                                                                  int64_t N, int n_chunks, int bits,
                                                                  uint32_t* __restrict__ qchunk_off) {
    __shared__ uint32_t part[QZ_SCAN_THREADS];
    const int tid = threadIdx.x;
    const int per = (n_chunks + QZ_SCAN_THREADS - 1) / QZ_SCAN_THREADS;   // chunks per thread
    const int c0 = tid * per;
    uint32_t sum = 0;
    for (int c = c0; c < c0 + per && c < n_chunks; ++c) {
        const int64_t t0 = (int64_t)c * CHUNK;
        for (int h = 0; h < 16; ++h) {
            const int64_t i = t0 + 16 * h;
            if (i < N) sum += qz_tile_bytes(srank[i], bits);
        }
    }
    part[tid] = sum;
    __syncthreads();
    // inclusive scan over the threads (Hillis-Steele)
    for (int off = 1; off < QZ_SCAN_THREADS; off <<= 1) {
        const uint32_t v = tid >= off ? part[tid - off] : 0u;
        __syncthreads();
        part[tid] += v;
        __syncthreads();
    }
    uint32_t run = tid ? part[tid - 1] : 0u;
    for (int c = c0; c < c0 + per && c < n_chunks; ++c) {
        qchunk_off[c] = run;
        const int64_t t0 = (int64_t)c * CHUNK;
        for (int h = 0; h < 16; ++h) {
            const int64_t i = t0 + 16 * h;
            if (i < N) run += qz_tile_bytes(srank[i], bits);
        }
    }
    if (tid == QZ_SCAN_THREADS - 1) qchunk_off[n_chunks] = part[tid];
}

struct QzParams {
    const uint16_t* coef[2];     // bf16 streams (K, V), [G][coef_stride]
    uint8_t* code[2];            // code streams (K, V), [G][q_stride] bytes
    const uint8_t* srank;
    const uint32_t* chunk_off;   // bf16 layout chunk bases (elements)
    const uint32_t* qchunk_off;  // quantised chunk bases (bytes)
    int64_t N, coef_stride, q_stride;
    int G, bits;
};

// One workgroup per (chunk, head, stream), its wave w taking tiles w, w + 4, w + 8, w + 12:
// the chunk's tile sizes are loaded once per wave and each tile runs in four steps that only the wave's own lanes share (its own LDS region,
// wave-scope fences): the bf16 tile rectangle into LDS, the 16 x KS group scales, every code
// (int8, [position][coordinate] for both streams), the packed dwords (each assembled by one
// lane from the fields it covers).  Element indices of a tile of size m are split into
// (row, column) by a float reciprocal: for f < 2048 and m <= 128, floor(f * (1/m) + 2^-10)
// is floor(f / m) exactly (the product errs by far less than 2^-10 and the fraction of f / m
// is at most 127/128 below an integer).
constexpr int QZ_WAVES = 4;
constexpr int QZ_VS = D + 1;                      // padded LDS row stride: no bank conflicts

__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int qz_div(int f, float inv) { return (int)(fmaf((float)f, inv, 0.0009765625f)); }

template <int QB>
__global__ __launch_bounds__(64 * QZ_WAVES) void qz_kernel(QzParams p, int total) {
    constexpr int QMAX = (1 << (QB - 1)) - 1;
    constexpr int VS = QZ_VS;
    __shared__ float val_s[QZ_WAVES][16 * VS];    // tile values, [position][coordinate]
    __shared__ float scl_s[QZ_WAVES][4 * 16];     // [group][position]
    __shared__ uint16_t sclh_s[QZ_WAVES][4 * 16]; // the same as binary16 bits
    __shared__ int8_t cod_s[QZ_WAVES][16 * VS];   // codes, [position][coordinate]
    const int wave = threadIdx.x >> 6, tid = threadIdx.x & 63;
    float* val = val_s[wave];
    float* scl = scl_s[wave];
    uint16_t* sclh = sclh_s[wave];
    int8_t* cod = cod_s[wave];
    const int item = blockIdx.x;                  // (chunk, head, stream); wave w takes tiles w, w + 4, ...
    if (item >= total) return;
    const int kv = item & 1;
    const int g = (item >> 1) % p.G;
    const int c = (item >> 1) / p.G;
    const int64_t t0 = (int64_t)c * CHUNK;
    const int T = (int)(p.N - t0 < CHUNK ? p.N - t0 : CHUNK);
    const int ntile = (T + 15) >> 4;
    // the chunk's tile sizes (lane h < 16 holds tile h's) and their prefix offsets
    const uint32_t mlane = tid < ntile ? (uint32_t)p.srank[t0 + 16 * tid] : 0u;
    uint32_t eo = p.chunk_off[c], bo = p.qchunk_off[c];
    const uint16_t* base_src = p.coef[kv] + (int64_t)g * p.coef_stride;
    uint8_t* base_dst = p.code[kv] + (int64_t)g * p.q_stride;
    for (int h = 0; h < wave; ++h) {
        const uint32_t m = (uint32_t)__builtin_amdgcn_readlane((int)mlane, h);
        eo += 16u * m;
        bo += qz_tile_bytes(m, QB);
    }
    for (int h = wave; h < ntile; h += QZ_WAVES) {
        const int mt = __builtin_amdgcn_readlane((int)mlane, h);
        const int mq = (mt + 7) & ~7, ks = (mt + 31) / 32;
        const uint16_t* src = base_src + eo;
        uint8_t* dst = base_dst + bo;
        // the offsets of this wave's next tile: past tiles h .. h + 3
        for (int k = h; k < h + QZ_WAVES && k < ntile; ++k) {
            const uint32_t m = (uint32_t)__builtin_amdgcn_readlane((int)mlane, k);
            eo += 16u * m;
            bo += qz_tile_bytes(m, QB);
        }
        const float inv_mt = 1.0f / (float)(mt > 0 ? mt : 1), inv_mq = 1.0f / (float)(mq > 0 ? mq : 1);
        // ---- 1. the tile rectangle (16 mt contiguous bf16: K rows of mt, or V rows of 16),
        //          16-byte loads scattered to [position][coordinate]; zeros up to mq
        for (int e8 = tid; e8 < 2 * mt; e8 += 64) {
            const u32x4 w = *reinterpret_cast<const u32x4*>(src + 8 * e8);
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int f = 8 * e8 + k;
                int i, j;
                if (kv == 0) { i = qz_div(f, inv_mt); j = f - i * mt; }
                else { j = f >> 4; i = f & 15; }
                val[i * VS + j] = (k & 1) ? bf_hi(w[k >> 1]) : bf_lo(w[k >> 1]);
            }
        }
        for (int e = tid; e < 16 * (mq - mt); e += 64) val[(e & 15) * VS + mt + (e >> 4)] = 0.f;
        wave_sync();
        // ---- 2. group scales: lane -> (group s, position i)
        if (tid < 16 * ks) {
            const int s = tid >> 4, i = tid & 15;
            float a[32];
#pragma unroll
            for (int u = 0; u < 32; ++u) {
                const int j = 32 * s + u;
                a[u] = j < mq ? fabsf(val[i * VS + j]) : 0.f;
            }
            float amax = 0.f;
#pragma unroll
            for (int u = 0; u < 32; ++u) amax = fmaxf(amax, a[u]);
            const _Float16 hs = (_Float16)__fdiv_rn(amax, (float)QMAX);   // nearest binary16
            scl[tid] = (float)hs;
            sclh[tid] = __builtin_bit_cast(uint16_t, hs);
        }
        wave_sync();
        // ---- 3. codes: element e -> position e & 15, coordinate e >> 4 (every lane busy)
        for (int e = tid; e < 16 * mq; e += 64) {
            const int i = e & 15, j = e >> 4;
            const float sc = scl[16 * (j >> 5) + i];
            int k = 0;
            if (sc != 0.f) {
                const float r = __builtin_rintf(__fdiv_rn(val[i * VS + j], sc));
                k = (int)fminf(fmaxf(r, (float)-QMAX), (float)QMAX);
            }
            cod[i * VS + j] = (int8_t)k;
        }
        wave_sync();
        // ---- 4. packed dwords: K code (i, j) is field i mq + j, V code (j, i) is field
        //          16 j + i; then the scales
        uint32_t* dw = reinterpret_cast<uint32_t*>(dst);      // tile start: 16-byte aligned
        const int nd = mq * QB / 2;
        constexpr int NF = (32 + QB - 1) / QB + 1;          // fields a dword can touch
        for (int d = tid; d < nd; d += 64) {
            uint32_t word = 0;
            const int ebeg = (32 * d) / QB, eend = (32 * d + 31) / QB;
            int8_t cv[NF];
#pragma unroll
            for (int u = 0; u < NF; ++u) {
                const int ee = ebeg + u <= eend ? ebeg + u : ebeg;   // in bounds; dropped below
                int i, j;
                if (kv == 0) { i = qz_div(ee, inv_mq); j = ee - i * mq; }
                else { j = ee >> 4; i = ee & 15; }
                cv[u] = cod[i * VS + j];
            }
#pragma unroll
            for (int u = 0; u < NF; ++u) {
                const int ee = ebeg + u;
                const uint32_t field = ee <= eend ? (uint32_t)(int)cv[u] & ((1u << QB) - 1u) : 0u;
                const int sh = QB * ee - 32 * d;
                word |= sh >= 0 ? (field << sh) : (field >> -sh);
            }
            dw[d] = word;
        }
        if (tid < 8 * ks) dw[nd + tid] = (uint32_t)sclh[2 * tid] | ((uint32_t)sclh[2 * tid + 1] << 16);
        wave_sync();                              // the wave's LDS is reused by its next tile
    }
}

// ----------------------------------------------------------------------------------------
size_t qcache_stride(const varrate_shape& sh, int bits) {
    const int64_t N = coded_count(sh);
    const int64_t n_chunks = (N + CHUNK - 1) / CHUNK;
    const int64_t B = coded_budget(sh);
    // a chunk's tile maxima sum to at most its ranks / 16 + 128, each tile pads up to 7
    // coordinates and holds at most 4 groups per position
    const int64_t bound = (int64_t)bits * B / 8 + n_chunks * (480LL * bits + 2048) + 64;
    return (size_t)((bound + 15) / 16 * 16);
}

hipError_t launch_quantize(const varrate_shape& sh, const varrate_cache& c, varrate_qcache& q, hipStream_t st) {
    const int64_t N = coded_count(sh);
    const int n_chunks = (int)((N + CHUNK - 1) / CHUNK);
    qz_scan_kernel<<<1, QZ_SCAN_THREADS, 0, st>>>(c.srank, N, n_chunks, q.bits, q.qchunk_off);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    QzParams p;
    p.coef[0] = (const uint16_t*)c.coef_k;
    p.coef[1] = (const uint16_t*)c.coef_v;
    p.code[0] = (uint8_t*)q.code_k;
    p.code[1] = (uint8_t*)q.code_v;
    p.srank = c.srank;
    p.chunk_off = c.chunk_off;
    p.qchunk_off = q.qchunk_off;
    p.N = N;
    p.coef_stride = c.coef_stride;
    p.q_stride = q.q_stride;
    p.G = sh.G;
    p.bits = q.bits;
    const int total = n_chunks * sh.G * 2;                      // (chunk, head, stream)
    const int grid = total;
    switch (q.bits) {
        case 3: qz_kernel<3><<<grid, 64 * QZ_WAVES, 0, st>>>(p, total); break;
        case 4: qz_kernel<4><<<grid, 64 * QZ_WAVES, 0, st>>>(p, total); break;
        case 8: qz_kernel<8><<<grid, 64 * QZ_WAVES, 0, st>>>(p, total); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace vr
