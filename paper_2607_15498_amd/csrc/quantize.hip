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
// qchunk_off; then one workgroup per (chunk, head, stream) writes its tiles (a wave per tile).
#include "vr_internal.h"

namespace vr {

constexpr int QZ_SCAN_THREADS = 1024;
constexpr int QZ_THREADS = 256;

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

template <int QB>
__global__ __launch_bounds__(QZ_THREADS) void qz_kernel(QzParams p) {
    constexpr int QMAX = (1 << (QB - 1)) - 1;
    __shared__ float scl[QZ_THREADS / 64][64];    // per wave: the tile's scales, [s][position]
    const int c = blockIdx.x / (2 * p.G);
    const int g = (blockIdx.x / 2) % p.G;
    const int kv = blockIdx.x & 1;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int64_t t0 = (int64_t)c * CHUNK;
    const int T = (int)(p.N - t0 < CHUNK ? p.N - t0 : CHUNK);
    // tile sizes of the chunk and their offsets in both layouts (every lane of every wave)
    uint32_t m[16], eoff[16], boff[16];
    uint32_t e = p.chunk_off[c], q = p.qchunk_off[c];
#pragma unroll
    for (int h = 0; h < 16; ++h) {
        m[h] = 16 * h < T ? (uint32_t)p.srank[t0 + 16 * h] : 0u;
        eoff[h] = e;
        boff[h] = q;
        e += 16u * m[h];
        q += qz_tile_bytes(m[h], QB);
    }
    const uint16_t* src = p.coef[kv] + (int64_t)g * p.coef_stride;
    uint8_t* dst = p.code[kv] + (int64_t)g * p.q_stride;
    // every wave takes 4 tiles (16 / 4), so the workgroup barriers below match up
    for (int h = wave; h < 16; h += QZ_THREADS / 64) {
        const int mt = (int)m[h];                   // wave-uniform; 0: no tile
        const int mq = (mt + 7) & ~7, ks = (mt + 31) / 32;
        const uint16_t* tile = src + eoff[h];
        uint8_t* out = dst + boff[h];
        // element (position i, coordinate j) of the bf16 tile rectangle
        auto val = [&](int i, int j) -> float {
            if (j >= mt) return 0.f;
            const int idx = kv == 0 ? i * mt + j : j * 16 + i;
            return bf16_to_f32(tile[idx]);
        };
        // ---- scales: lane -> group (s, i) = (lane / 16, lane % 16)
        {
            const int s = lane >> 4, i = lane & 15;
            float sc = 0.f;
            if (s < ks) {
                float amax = 0.f;
                for (int j = 32 * s; j < 32 * s + 32; ++j) amax = fmaxf(amax, fabsf(val(i, j)));
                const float ratio = __fdiv_rn(amax, (float)QMAX);
                const _Float16 hs = (_Float16)ratio;           // nearest binary16, ties to even
                sc = (float)hs;
                reinterpret_cast<uint16_t*>(out + 2 * mq * QB)[16 * s + i] = __builtin_bit_cast(uint16_t, hs);
            }
            scl[wave][lane] = sc;
        }
        __syncthreads();
        // ---- codes: lane -> output bytes lane, lane + 64, ...
        const int nbytes = 2 * mq * QB;
        for (int B = lane; B < nbytes; B += 64) {
            uint32_t byte = 0;
            const int ebeg = (8 * B) / QB, eend = (8 * B + 7) / QB;
            for (int ee = ebeg; ee <= eend; ++ee) {
                int i, j;
                if (kv == 0) { i = ee / mq; j = ee % mq; }
                else { j = ee >> 4; i = ee & 15; }
                const float sc = scl[wave][16 * (j >> 5) + i];
                int k = 0;
                if (sc != 0.f) {
                    float r = __builtin_rintf(__fdiv_rn(val(i, j), sc));
                    r = fminf(fmaxf(r, (float)-QMAX), (float)QMAX);
                    k = (int)r;
                }
                const uint32_t field = (uint32_t)k & ((1u << QB) - 1u);
                const int sh = QB * ee - 8 * B;             // field position relative to the byte
                byte |= sh >= 0 ? (field << sh) : (field >> -sh);
            }
            out[B] = (uint8_t)(byte & 0xFFu);
        }
        __syncthreads();
    }
}

// ----------------------------------------------------------------------------------------
size_t qcache_stride(const varrate_shape& sh, int bits) {
    const int64_t N = sh.n - sh.w;
    const int64_t n_chunks = (N + CHUNK - 1) / CHUNK;
    const int64_t B = varrate_coded_budget(sh.n, sh.d, sh.w, sh.kappa_pct);
    // a chunk's tile maxima sum to at most its ranks / 16 + 128, each tile pads up to 7
    // coordinates and holds at most 4 groups per position
    const int64_t bound = (int64_t)bits * B / 8 + n_chunks * (480LL * bits + 2048) + 64;
    return (size_t)((bound + 15) / 16 * 16);
}

hipError_t launch_quantize(const varrate_shape& sh, const varrate_cache& c, varrate_qcache& q, hipStream_t st) {
    const int64_t N = sh.n - sh.w;
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
    const unsigned grid = (unsigned)(n_chunks * sh.G * 2);
    switch (q.bits) {
        case 3: qz_kernel<3><<<grid, QZ_THREADS, 0, st>>>(p); break;
        case 4: qz_kernel<4><<<grid, QZ_THREADS, 0, st>>>(p); break;
        case 8: qz_kernel<8><<<grid, QZ_THREADS, 0, st>>>(p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace vr
