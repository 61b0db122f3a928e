// Basis projection + nested truncation + packing (Sec. 3.3 Eq. (6), Algorithm 1), gfx950.
//
// One workgroup per (group of CPW chunks, KV head g, K|V), one workgroup per CU: CPW = 8, or
// 4 or 2 when that leaves fewer than 256 workgroups (short contexts, few heads).  The
// storage order of every chunk (srank, sidx: rank descending, index ascending) comes with
// the ranks from the allocation.
//   1. The basis P (fp32) is split into bf16 hi + lo parts once per workgroup and kept in
//      LDS in MFMA-fragment order (64 KB), so every product is P_hi x + P_lo x with exact
//      bf16 x (fp32 x adds P_hi x_lo): about 2^-16 relative error before storage rounding.
//   2. A wave takes 16-position tiles of the stored order (the tiles of a chunk rotate over
//      the waves from chunk to chunk) and computes only the 16-row coefficient blocks below
//      the tile's size m (its largest rank, its first position's).  The tile is stored as
//      a rectangle with zeros past each position's rank: K as 16 rows of m coordinates (the
//      C tile gives each lane four consecutive coordinates of one position), V as m rows of
//      16 positions (C^T by swapped operands: four consecutive positions at one coordinate).
//   3. The tile loop is fully unrolled with a fixed number of loads per tile: the layout rows
//      of tile k + 4 and the token rows of tile k + 3 are requested while tile k is computed,
//      and tile k's coefficients stay in registers until the data of tile k + 1 has landed.
//      Vector-memory loads and stores share one completion counter, so a wait then never
//      covers stores issued just before it.  With three tiles of token rows in flight per
//      wave, eight waves keep about 96 KB of loads in flight per CU.
// Workgroups of chunk group 0 also copy the window rows into the exact slots.
#include "vr_internal.h"

namespace vr {

constexpr int PJ_THREADS = 512;                       // 8 waves
constexpr int PJ_WAVES = PJ_THREADS / 64;
constexpr int PJ_CPW = 8;                             // chunks per workgroup (at most)
constexpr int PJ_HT = 16;                             // tokens per tile
constexpr int PJ_TPC = CHUNK / PJ_HT;                 // tiles per chunk
constexpr int PJ_FRAGS = 8 * 4;                       // (16-row block a, 32-col step s) pairs
// token rows are requested XD tiles ahead (fp32 rows are twice as large: one tile less),
// layout rows one tile further
template <bool F32> __host__ __device__ constexpr int pj_xd() { return F32 ? 2 : 3; }
static_assert(2 * PJ_TPC % PJ_WAVES == 0, "whole tiles per wave for 2, 4 and 8 chunks per workgroup");

constexpr size_t PJ_FRAG_BYTES = (size_t)PJ_FRAGS * 64 * 16 * 2;
// the basis fragments (hi, lo), then the workgroup's chunk offsets
static inline size_t project_smem_bytes() { return PJ_FRAG_BYTES + 64; }

// Layout rows of one tile, per lane: srank of slots 4 lane .. 4 lane + 3 of the chunk, and
// the token of slot 16 h + (lane % 16).
struct PjMeta {
    uint32_t quad;
    uint32_t tok;
};

template <bool F32>
struct PjX {                                           // B fragments of the tile's 16 tokens
    u32x4 a[4];
    u32x4 b[F32 ? 4 : 1];                              // fp32: second half of each 8-element run
};

// Coefficients of one tile held for the late store, and where they go.  K lanes hold four
// consecutive coordinates of one position, V lanes four consecutive positions at one
// coordinate; entries past a position's rank are already zero.
template <bool F32>
struct PjOut {
    uint32_t v[8][F32 ? 4 : 2];                        // per 16-row block: 4 values (packed bf16)
    int na;                                            // blocks computed (uniform)
    int m;                                             // the tile's size: its largest rank (uniform)
    uint32_t off;                                      // the tile's first element in the head stream
};

__device__ __forceinline__ void pj_tile_of(int k, int wave, int c0, int& c, int& h) {
    const int item = k * PJ_WAVES + wave;
    const int cc = item / PJ_TPC;
    h = (item + cc) % PJ_TPC;
    c = c0 + cc;
}

// Loads with clamped addresses only: their number per tile is fixed.
__device__ __forceinline__ PjMeta pj_load_meta(int k, int wave, int c0, int n_chunks, int64_t N,
                                               const uint8_t* __restrict__ srank,
                                               const uint32_t* __restrict__ sidx) {
    const int lane = threadIdx.x & 63;
    int c, h;
    pj_tile_of(k, wave, c0, c, h);
    const bool live = c < n_chunks;
    const int64_t t0 = live ? (int64_t)c * CHUNK : 0;
    const int64_t T = live ? (N - t0 < CHUNK ? N - t0 : CHUNK) : 0;
    // srank is padded to a multiple of 64 bytes: a quad that starts before N stays inside
    const int64_t qi = 4 * lane < T ? t0 + 4 * lane : 0;
    const int64_t si = PJ_HT * h + (lane & 15) < T ? t0 + PJ_HT * h + (lane & 15) : 0;
    PjMeta m;
    m.quad = *reinterpret_cast<const uint32_t*>(srank + qi);
    m.tok = sidx[si];
    return m;
}

// Make the compiler wait for these registers here (its waits go to the first use).
__device__ __forceinline__ void pj_ready(uint32_t v) { asm volatile("" ::"v"(v)); }
template <bool F32>
__device__ __forceinline__ void pj_ready(const PjX<F32>& x) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        asm volatile("" ::"v"(x.a[s]));
        if constexpr (F32) asm volatile("" ::"v"(x.b[s]));
    }
}

template <bool F32>
__device__ __forceinline__ void pj_load_x(PjX<F32>& x, const void* X, uint32_t tok, int64_t N, int G,
                                          int g) {
    const int grp = (threadIdx.x & 63) >> 4;
    const int64_t t = (int64_t)tok < N ? (int64_t)tok : N - 1;   // a valid row whatever sidx holds
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const int64_t e0 = (t * G + g) * D + 32 * s + 8 * grp;
        if constexpr (!F32) {
            x.a[s] = load16((const uint16_t*)X + e0);
        } else {
            x.a[s] = load16((const float*)X + e0);
            x.b[s] = load16((const float*)X + e0 + 4);
        }
    }
}

// Tile k: its size and place from the layout rows, then the coefficient blocks into `o`:
// C = P x (K: lane -> position col, coordinates 16 a + 4 grp ..) or C^T = x^T P^T (V: lane
// -> coordinate 16 a + col, positions 4 grp ..), with zeros past each position's rank.
template <bool F32>
__device__ __forceinline__ void pj_compute(PjOut<F32>& o, const PjMeta& m, const PjX<F32>& x, int k,
                                           int wave, int c0, int n_chunks, int64_t N, bool is_v,
                                           const uint32_t* cbase,
                                           int64_t coef_stride, const u32x4* frag_hi,
                                           const u32x4* frag_lo) {
    const int lane = threadIdx.x & 63, col = lane & 15, grp = lane >> 4;
    int c, h;
    pj_tile_of(k, wave, c0, c, h);
    const bool live = c < n_chunks;
    const int64_t t0 = (int64_t)c * CHUNK;
    const int T = live ? (int)(N - t0 < CHUNK ? N - t0 : CHUNK) : 0;
    // bytes past the chunk's end weigh nothing (absent positions: rank 0)
    uint32_t quad = m.quad;
    const int nv = T - 4 * lane;
    quad = nv >= 4 ? quad : (nv <= 0 ? 0u : quad & ((1u << (8 * nv)) - 1u));
    // tile sizes: the first rank of every 16 positions (byte 0 of quads 0, 4, 8, ..), and
    // their prefix up to tile h
    uint32_t incl = (lane & 3) == 0 ? (quad & 0xFF) : 0u;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_up(incl, off, 64);
        if (lane >= off) incl += y;
    }
    const int mt = __builtin_amdgcn_readfirstlane((int)(__shfl(quad, 4 * h, 64) & 0xFF));
    const uint32_t before = __builtin_amdgcn_readfirstlane(__shfl(incl, 4 * h, 64)) - (uint32_t)mt;
    const uint32_t base = live ? cbase[c - c0] : 0u;
    o.off = __builtin_amdgcn_readfirstlane(base + 16u * before);
    o.m = mt;
    // the tile stays inside the head's stream whatever the layout tables hold
    const bool fits = (int64_t)o.off + 16 * (int64_t)mt <= coef_stride;
    int na = (mt + 15) >> 4;
    na = live && fits ? (na < D / 16 ? na : D / 16) : 0;
    o.na = __builtin_amdgcn_readfirstlane(na);
    // ranks: K -> this lane's position 16 h + col; V -> positions 16 h + 4 grp .. + 3
    const uint32_t qk = __shfl(quad, 4 * h + (col >> 2), 64);
    const int rk = (int)((qk >> (8 * (col & 3))) & 0xFF);
    const uint32_t qv = __shfl(quad, 4 * h + grp, 64);

    u32x4 xh[4], xl[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        if constexpr (!F32) {
            xh[s] = x.a[s];
            xl[s] = u32x4{0, 0, 0, 0};
        } else {
            float x8[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                x8[e] = __uint_as_float(x.a[s][e]);
                x8[4 + e] = __uint_as_float(x.b[s][e]);
            }
            split8(x8, xh[s], xl[s]);
        }
    }
#pragma unroll
    for (int a = 0; a < D / 16; ++a) {
        if (a >= o.na) break;
        f32x4 acc = {0, 0, 0, 0};
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const u32x4 ph = frag_hi[(a * 4 + s) * 64 + lane];
            const u32x4 pl = frag_lo[(a * 4 + s) * 64 + lane];
            if (!is_v) {
                acc = mfma(ph, xh[s], acc);
                acc = mfma(pl, xh[s], acc);
                if constexpr (F32) acc = mfma(ph, xl[s], acc);
            } else {
                acc = mfma(xh[s], ph, acc);
                acc = mfma(xh[s], pl, acc);
                if constexpr (F32) acc = mfma(xl[s], ph, acc);
            }
        }
        // zeros past each position's rank
        float val[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int j = is_v ? 16 * a + col : 16 * a + 4 * grp + v;
            const int r = is_v ? (int)((qv >> (8 * v)) & 0xFF) : rk;
            val[v] = j < r ? acc[v] : 0.f;
        }
        if constexpr (F32) {
#pragma unroll
            for (int v = 0; v < 4; ++v) o.v[a][v] = __float_as_uint(val[v]);
        } else {
            o.v[a][0] = cvt_bf16x2(val[0], val[1]);
            o.v[a][1] = cvt_bf16x2(val[2], val[3]);
        }
    }
}

// Store a computed tile.  K: rows of m coordinates, the lane's four coordinates at once
// unless the row ends inside them.  V: coordinate rows of 16 positions, the lane's four
// positions at once (aligned: tiles start at multiples of 16 elements).
template <bool F32>
__device__ __forceinline__ void pj_store(const PjOut<F32>& o, bool is_v, void* __restrict__ coef) {
    const int lane = threadIdx.x & 63, col = lane & 15, grp = lane >> 4;
#pragma unroll
    for (int a = 0; a < D / 16; ++a) {
        if (a >= o.na) break;
        if (is_v) {
            const int j = 16 * a + col;
            if (j < o.m) {
                const int64_t e = (int64_t)o.off + 16 * j + 4 * grp;
                if constexpr (F32) __builtin_memcpy((float*)coef + e, &o.v[a][0], 16);
                else {
                    const uint2 pk = make_uint2(o.v[a][0], o.v[a][1]);
                    *reinterpret_cast<uint2*>((uint16_t*)coef + e) = pk;
                }
            }
        } else {
            const int j0 = 16 * a + 4 * grp;
            const int64_t e = (int64_t)o.off + (int64_t)col * o.m + j0;
            if constexpr (F32) {
                float* p = (float*)coef + e;
                if (j0 + 4 <= o.m) {
                    __builtin_memcpy(p, &o.v[a][0], 16);
                } else {
#pragma unroll
                    for (int v = 0; v < 3; ++v)
                        if (j0 + v < o.m) p[v] = __uint_as_float(o.v[a][v]);
                }
            } else {
                uint16_t* p = (uint16_t*)coef + e;
                if (j0 + 4 <= o.m) {
                    const uint2 pk = make_uint2(o.v[a][0], o.v[a][1]);
                    __builtin_memcpy(p, &pk, 8);
                } else {
                    if (j0 < o.m) p[0] = (uint16_t)o.v[a][0];
                    if (j0 + 1 < o.m) p[1] = (uint16_t)(o.v[a][0] >> 16);
                    if (j0 + 2 < o.m) p[2] = (uint16_t)o.v[a][1];
                }
            }
        }
    }
}

template <bool F32, bool IS_V, int CPW>
__device__ __forceinline__ void project_body(
    const void* __restrict__ K, const void* __restrict__ V, const float* __restrict__ PK,
    const float* __restrict__ PV, int64_t N, int G, int w, const uint8_t* __restrict__ srank,
    const uint32_t* __restrict__ sidx, const uint32_t* __restrict__ csum, uint32_t* __restrict__ chunk_off,
    int n_chunks, void* __restrict__ coef_k, void* __restrict__ coef_v, int64_t coef_stride,
    void* __restrict__ k_exact, void* __restrict__ v_exact, int64_t cap, uint8_t* smem) {
    u32x4* frag_hi = reinterpret_cast<u32x4*>(smem);
    u32x4* frag_lo = frag_hi + PJ_FRAGS * 64;
    uint32_t* cbase = reinterpret_cast<uint32_t*>(smem + PJ_FRAG_BYTES);

    const int g = blockIdx.y, kv = IS_V ? 1 : 0;
    const void* X = kv ? V : K;
    // this head's stream
    void* coef = (uint8_t*)(kv ? coef_v : coef_k) + (int64_t)g * coef_stride * (F32 ? 4 : 2);
    constexpr bool is_v = IS_V;
    const float* P = (kv ? PV : PK) + (int64_t)g * D * D;
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    constexpr int PJ_ITERS = CPW * PJ_TPC / PJ_WAVES;   // tiles per wave
    const int c0 = blockIdx.x * CPW;

    // offsets of this workgroup's chunks (wave 0): read from the chunk table, or (csum given)
    // scanned from the chunk sizes.  The sizes of the first 512 chunks are requested here, ahead
    // of every other load (clamped addresses, masked values).
    const int lane0 = tid & 63, cown = c0 + lane0;
    const bool own = lane0 < CPW && cown < n_chunks;
    uint32_t cs_v[8], cs_sz = 0;
    if (csum && wave == 0) {
        cs_sz = csum[own ? cown : 0];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int i = 64 * j + lane0;
            cs_v[j] = csum[i < c0 ? i : 0];
        }
    }

    constexpr int PJ_XD = pj_xd<F32>(), PJ_MD = PJ_XD + 1;
    // ---- layout rows of the first PJ_MD tiles and the basis, all requested at once
    PjMeta m[PJ_ITERS];
    PjX<F32> x[PJ_ITERS];
    PjOut<F32> o;
#pragma unroll
    for (int k = 0; k < PJ_MD && k < PJ_ITERS; ++k) m[k] = pj_load_meta(k, wave, c0, n_chunks, N, srank, sidx);
    constexpr int PER = PJ_FRAGS * 64 / PJ_THREADS;   // fragment entries per thread
    u32x4 p0[PER], p1[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        // fragment f = a * 4 + s, lane l -> row 16a + l%16, cols 32s + 8(l/16)
        const int idx = tid + e * PJ_THREADS;
        const int f = idx >> 6, l = idx & 63;
        const float* src = P + (16 * (f >> 2) + (l & 15)) * D + 32 * (f & 3) + 8 * (l >> 4);
        p0[e] = load16(src);
        p1[e] = load16(src + 4);
    }
    // token rows of the first PJ_XD tiles as soon as their layout rows are in
#pragma unroll
    for (int k = 0; k < PJ_XD && k < PJ_ITERS; ++k) pj_load_x<F32>(x[k], X, m[k].tok, N, G, g);
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        float v[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) { v[i] = __uint_as_float(p0[e][i]); v[4 + i] = __uint_as_float(p1[e][i]); }
        split8(v, frag_hi[tid + e * PJ_THREADS], frag_lo[tid + e * PJ_THREADS]);
    }
    if (wave == 0) {
        if (csum) {
            // every earlier chunk's size summed, the group's own scanned across lanes; the
            // workgroups of head 0's K half write the table
            uint32_t pre = 0;
#pragma unroll
            for (int j = 0; j < 8; ++j) pre += 64 * j + lane0 < c0 ? cs_v[j] : 0u;
            for (int i0 = 8 * 64; i0 < c0; i0 += 8 * 64) {
                uint32_t v[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int i = i0 + 64 * j + lane0;
                    v[j] = csum[i < c0 ? i : 0];
                }
#pragma unroll
                for (int j = 0; j < 8; ++j) pre += i0 + 64 * j + lane0 < c0 ? v[j] : 0u;
            }
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) pre += __shfl_xor(pre, off, 64);
            const uint32_t sz = own ? cs_sz : 0u;
            uint32_t incl = sz;
#pragma unroll
            for (int off = 1; off < CPW; off <<= 1) {
                const uint32_t y = __shfl_up(incl, off, 64);
                if (lane0 >= off) incl += y;
            }
            const uint32_t base = pre + incl - sz;
            if (lane0 < CPW) cbase[lane0] = base;
            if (blockIdx.y == 0 && blockIdx.z == 0 && own) {
                chunk_off[cown] = base;
                if (cown == n_chunks - 1) chunk_off[n_chunks] = base + sz;
            }
        } else if (lane0 < CPW) {
            cbase[lane0] = own ? chunk_off[cown] : 0u;
        }
    }
    __syncthreads();

    // ---- tile loop (fully unrolled: every load count is fixed).  The top of tile k waits for
    // its token rows and tile k + PJ_XD's layout rows, which leaves the token rows of tiles
    // k + 1 .. k + PJ_XD - 1 in flight; only then do tile k - 1's stores go out, followed by
    // the next requests.
#pragma unroll
    for (int k = 0; k < PJ_ITERS; ++k) {
        pj_ready(x[k]);
        if (k + PJ_XD < PJ_ITERS) pj_ready(m[k + PJ_XD].tok);
        if (k > 0) pj_store<F32>(o, is_v, coef);                         // tile k - 1, late
        if (k + PJ_MD < PJ_ITERS) m[k + PJ_MD] = pj_load_meta(k + PJ_MD, wave, c0, n_chunks, N, srank, sidx);
        if (k + PJ_XD < PJ_ITERS) pj_load_x<F32>(x[k + PJ_XD], X, m[k + PJ_XD].tok, N, G, g);
        pj_compute<F32>(o, m[k], x[k], k, wave, c0, n_chunks, N, is_v, cbase, coef_stride,
                        frag_hi, frag_lo);
    }
    pj_store<F32>(o, is_v, coef);

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

// K (blockIdx.z = 0) and V (blockIdx.z = 1) in one launch; their stores differ, so each
// half runs its own instance of the body.
template <bool F32, int CPW>
__global__ __launch_bounds__(PJ_THREADS, 1) void project_kernel(
    const void* __restrict__ K, const void* __restrict__ V, const float* __restrict__ PK,
    const float* __restrict__ PV, int64_t N, int G, int w, const uint8_t* __restrict__ srank,
    const uint32_t* __restrict__ sidx, const uint32_t* __restrict__ csum, uint32_t* __restrict__ chunk_off,
    int n_chunks, void* __restrict__ coef_k, void* __restrict__ coef_v, int64_t coef_stride,
    void* __restrict__ k_exact, void* __restrict__ v_exact, int64_t cap) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    if (blockIdx.z == 0)
        project_body<F32, false, CPW>(K, V, PK, PV, N, G, w, srank, sidx, csum, chunk_off, n_chunks, coef_k,
                                      coef_v, coef_stride, k_exact, v_exact, cap, smem);
    else
        project_body<F32, true, CPW>(K, V, PK, PV, N, G, w, srank, sidx, csum, chunk_off, n_chunks, coef_k,
                                     coef_v, coef_stride, k_exact, v_exact, cap, smem);
}

template <bool F32, int CPW>
static hipError_t project_launch(const varrate_shape& sh, const void* K, const void* V, const float* PK,
                                 const float* PV, varrate_cache& c, hipStream_t st, const uint32_t* chunk_sizes,
                                 int n_chunks) {
    const int64_t N = sh.n - sh.w;
    const size_t lds = project_smem_bytes();
    hipError_t e = ensure_lds_limit((const void*)project_kernel<F32, CPW>, lds);
    if (e != hipSuccess) return e;
    dim3 grid((n_chunks + CPW - 1) / CPW, sh.G, 2);
    project_kernel<F32, CPW><<<grid, PJ_THREADS, lds, st>>>(
        K, V, PK, PV, N, sh.G, sh.w, c.srank, c.sidx, chunk_sizes, c.chunk_off, n_chunks, c.coef_k, c.coef_v,
        c.coef_stride, c.k_exact, c.v_exact, c.cap);
    return hipGetLastError();
}

template <bool F32>
static hipError_t project_launch_cpw(const varrate_shape& sh, const void* K, const void* V, const float* PK,
                                     const float* PV, varrate_cache& c, hipStream_t st,
                                     const uint32_t* chunk_sizes, int n_chunks) {
    // the most chunks per workgroup that still gives every CU a workgroup
    auto wgs = [&](int cpw) { return (int64_t)((n_chunks + cpw - 1) / cpw) * sh.G * 2; };
    if (wgs(8) >= 256) return project_launch<F32, 8>(sh, K, V, PK, PV, c, st, chunk_sizes, n_chunks);
    if (wgs(4) >= 256) return project_launch<F32, 4>(sh, K, V, PK, PV, c, st, chunk_sizes, n_chunks);
    return project_launch<F32, 2>(sh, K, V, PK, PV, c, st, chunk_sizes, n_chunks);
}

hipError_t launch_project(const varrate_shape& sh, const void* K, const void* V, const float* PK,
                          const float* PV, varrate_cache& c, hipStream_t st, const uint32_t* chunk_sizes) {
    const int64_t N = sh.n - sh.w;
    const int n_chunks = (int)((N + CHUNK - 1) / CHUNK);
    return sh.dtype == VARRATE_BF16 ? project_launch_cpw<false>(sh, K, V, PK, PV, c, st, chunk_sizes, n_chunks)
                                    : project_launch_cpw<true>(sh, K, V, PK, PV, c, st, chunk_sizes, n_chunks);
}

}  // namespace vr
