// Basis projection + nested truncation + packing (Sec. 3.3 Eq. (6), Algorithm 1), gfx950.
//
// One workgroup per (group of PJ_CPW chunks, KV head g, K|V).  The basis P (fp32) is split
// into bf16 hi + lo parts once per workgroup and kept in LDS in MFMA-fragment order (64 KB),
// so every product is P_hi x + P_lo x with exact bf16 x (fp32 x adds P_hi x_lo): about 2^-16
// relative error before the storage rounding.  Work items are super-tiles of 32 stored
// tokens; a super-tile only computes the 16-row coefficient blocks j < its largest rank
// (tokens are stored rank-descending inside a chunk, so the first token has the largest
// rank).  The C tile (16 coefficients x 16 tokens) is written straight into the ragged
// packed rows.  Workgroups of chunk group 0 also copy the window rows into the exact slots.
#include "vr_internal.h"

namespace vr {

constexpr int PJ_THREADS = 512;     // 8 waves
constexpr int PJ_CPW = 4;           // chunks per workgroup
constexpr int PJ_FRAGS = 8 * 4;     // (16-row block a, 32-col step s) pairs

template <bool F32>
__global__ __launch_bounds__(PJ_THREADS) void project_kernel(
    const void* __restrict__ K, const void* __restrict__ V, const float* __restrict__ PK,
    const float* __restrict__ PV, int64_t n, int64_t N, int G, int w,
    const uint8_t* __restrict__ srank, const uint32_t* __restrict__ sidx,
    const uint32_t* __restrict__ chunk_off, int n_chunks, void* __restrict__ coef_k,
    void* __restrict__ coef_v, int64_t coef_stride, void* __restrict__ k_exact,
    void* __restrict__ v_exact, int64_t cap) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    u32x4* frag_hi = reinterpret_cast<u32x4*>(smem);                       // [32][64]
    u32x4* frag_lo = frag_hi + PJ_FRAGS * 64;                              // [32][64]
    uint32_t* s_tok = reinterpret_cast<uint32_t*>(frag_lo + PJ_FRAGS * 64); // [CPW][256]
    uint16_t* s_off = reinterpret_cast<uint16_t*>(s_tok + PJ_CPW * CHUNK);  // [CPW][256]
    uint8_t* s_rank = reinterpret_cast<uint8_t*>(s_off + PJ_CPW * CHUNK);   // [CPW][256]
    __shared__ uint32_t s_base[PJ_CPW];
    __shared__ int s_T[PJ_CPW];
    __shared__ int s_tiles[PJ_CPW + 1];

    const int g = blockIdx.y, kv = blockIdx.z;
    const void* X = kv ? V : K;
    const float* P = (kv ? PV : PK) + (int64_t)g * D * D;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int c0 = blockIdx.x * PJ_CPW;

    // ---- basis fragments: fragment f = a * 4 + s, lane l -> row 16a + l%16, cols 32s + 8(l/16)
    for (int idx = tid; idx < PJ_FRAGS * 64; idx += PJ_THREADS) {
        const int f = idx >> 6, l = idx & 63;
        const int a = f >> 2, s = f & 3;
        const float* src = P + (16 * a + (l & 15)) * D + 32 * s + 8 * (l >> 4);
        float x[8];
        u32x4 p0 = load16(src), p1 = load16(src + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) { x[e] = __uint_as_float(p0[e]); x[4 + e] = __uint_as_float(p1[e]); }
        split8(x, frag_hi[idx], frag_lo[idx]);
    }
    // ---- chunk slot tables
    for (int cc = 0; cc < PJ_CPW; ++cc) {
        const int c = c0 + cc;
        const int64_t t0 = (int64_t)c * CHUNK;
        const int T = c < n_chunks ? (int)((N - t0) < CHUNK ? (N - t0) : CHUNK) : 0;
        if (tid == 0) {
            s_T[cc] = T;
            s_base[cc] = c < n_chunks ? chunk_off[c] : 0;
        }
        for (int i = tid; i < CHUNK; i += PJ_THREADS) {
            s_rank[cc * CHUNK + i] = i < T ? srank[t0 + i] : 0;
            s_tok[cc * CHUNK + i] = i < T ? sidx[t0 + i] : 0;
        }
    }
    __syncthreads();
    // local offsets: wave cc scans chunk cc (4 entries per lane)
    if (wave < PJ_CPW) {
        const int cc = wave;
        uint32_t r[4], loc = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) { r[e] = s_rank[cc * CHUNK + 4 * lane + e]; loc += r[e]; }
        uint32_t x = loc;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            uint32_t y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        uint32_t pre = x - loc;
#pragma unroll
        for (int e = 0; e < 4; ++e) { s_off[cc * CHUNK + 4 * lane + e] = (uint16_t)pre; pre += r[e]; }
    }
    if (tid == 0) {
        int acc = 0;
        for (int cc = 0; cc < PJ_CPW; ++cc) { s_tiles[cc] = acc; acc += (s_T[cc] + 31) / 32; }
        s_tiles[PJ_CPW] = acc;
    }
    __syncthreads();

    // ---- projection of 32-token super-tiles
    const int ntiles = s_tiles[PJ_CPW];
    const int grp = lane >> 4, col = lane & 15;
    for (int tile = wave; tile < ntiles; tile += PJ_THREADS / 64) {
        int cc = 0;
        while (tile >= s_tiles[cc + 1]) ++cc;
        const int i0 = (tile - s_tiles[cc]) * 32;
        const int T = s_T[cc];
        const int rmax = s_rank[cc * CHUNK + i0];
        const int na = (rmax + 15) >> 4;
        // token fragments: half hb covers stored slots i0 + 16 hb + col
        u32x4 xh[2][4], xl[2][4];
        int r_of[2], o_of[2];
#pragma unroll
        for (int hb = 0; hb < 2; ++hb) {
            const int i = i0 + 16 * hb + col;
            const bool ok = i < T;
            r_of[hb] = ok ? s_rank[cc * CHUNK + i] : 0;
            o_of[hb] = ok ? s_off[cc * CHUNK + i] : 0;
            const int64_t t = ok ? (int64_t)s_tok[cc * CHUNK + i] : 0;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int64_t e0 = (t * G + g) * D + 32 * s + 8 * grp;
                if constexpr (!F32) {
                    xh[hb][s] = ok ? load16((const uint16_t*)X + e0) : u32x4{0, 0, 0, 0};
                    xl[hb][s] = u32x4{0, 0, 0, 0};
                } else {
                    float x[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                    if (ok) {
                        u32x4 p0 = load16((const float*)X + e0), p1 = load16((const float*)X + e0 + 4);
#pragma unroll
                        for (int e = 0; e < 4; ++e) { x[e] = __uint_as_float(p0[e]); x[4 + e] = __uint_as_float(p1[e]); }
                    }
                    split8(x, xh[hb][s], xl[hb][s]);
                }
            }
        }
        const int64_t out0 = (int64_t)g * coef_stride + s_base[cc];
        for (int a = 0; a < na; ++a) {
            u32x4 ph[4], pl[4];
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                ph[s] = frag_hi[(a * 4 + s) * 64 + lane];
                pl[s] = frag_lo[(a * 4 + s) * 64 + lane];
            }
#pragma unroll
            for (int hb = 0; hb < 2; ++hb) {
                f32x4 c = {0, 0, 0, 0};
#pragma unroll
                for (int s = 0; s < 4; ++s) {
                    c = mfma(ph[s], xh[hb][s], c);
                    c = mfma(pl[s], xh[hb][s], c);
                    if constexpr (F32) c = mfma(ph[s], xl[hb][s], c);
                }
                // C: lane -> token column (slot i0 + 16hb + col), rows j = 16a + 4grp + v
                const int r = r_of[hb];
                const int64_t dst = out0 + o_of[hb];
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int j = 16 * a + 4 * grp + v;
                    if (j < r) {
                        if constexpr (F32) ((float*)(kv ? coef_v : coef_k))[dst + j] = c[v];
                        else ((uint16_t*)(kv ? coef_v : coef_k))[dst + j] = (uint16_t)f32_to_bf16(c[v]);
                    }
                }
            }
        }
    }

    // ---- exact window rows (chunk group 0 only)
    if (blockIdx.x == 0) {
        const int es = F32 ? 4 : 2;
        const uint8_t* src = (const uint8_t*)X;
        uint8_t* dst = (uint8_t*)(kv ? v_exact : k_exact);
        const int per_row = D * es / 16;   // 16-byte pieces per row
        for (int idx = tid; idx < w * per_row; idx += PJ_THREADS) {
            const int e = idx / per_row, p = idx % per_row;
            const int64_t so = (((N + e) * G + g) * D) * es + p * 16;
            const int64_t d0 = (((int64_t)g * cap + e) * D) * es + p * 16;
            *reinterpret_cast<u32x4*>(dst + d0) = *reinterpret_cast<const u32x4*>(src + so);
        }
    }
}

size_t project_lds_bytes() {
    return (size_t)PJ_FRAGS * 64 * 16 * 2 + (size_t)PJ_CPW * CHUNK * (4 + 2 + 1);
}

hipError_t launch_project(const varrate_shape& sh, const void* K, const void* V, const float* PK,
                          const float* PV, varrate_cache& c, hipStream_t st) {
    const int64_t N = sh.n - sh.w;
    const int n_chunks = (int)((N + CHUNK - 1) / CHUNK);
    dim3 grid((n_chunks + PJ_CPW - 1) / PJ_CPW, sh.G, 2);
    const size_t lds = project_lds_bytes();
    if (sh.dtype == VARRATE_BF16) {
        hipError_t e = hipFuncSetAttribute((const void*)project_kernel<false>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        project_kernel<false><<<grid, PJ_THREADS, lds, st>>>(
            K, V, PK, PV, sh.n, N, sh.G, sh.w, c.srank, c.sidx, c.chunk_off, n_chunks, c.coef_k,
            c.coef_v, c.coef_stride, c.k_exact, c.v_exact, c.cap);
    } else {
        hipError_t e = hipFuncSetAttribute((const void*)project_kernel<true>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
        project_kernel<true><<<grid, PJ_THREADS, lds, st>>>(
            K, V, PK, PV, sh.n, N, sh.G, sh.w, c.srank, c.sidx, c.chunk_off, n_chunks, c.coef_k,
            c.coef_v, c.coef_stride, c.k_exact, c.v_exact, c.cap);
    }
    return hipGetLastError();
}

}  // namespace vr
