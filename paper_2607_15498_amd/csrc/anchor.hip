// Residual codec with strided anchors (Sec. 3.1 "Residual codec", Eq. (2); Algorithm 1):
// compress-side kernels, gfx950.
//
// Anchors are the prefix tokens t = a delta (a = 0 .. na - 1, t < N); they and the window
// stay exact.  Coded token number i (the prefix tokens that are not anchors, in order) is
// token t(i) = i + i / (delta - 1) + 1.  Each coded token is coded as its residual to the mean
// of its c = 4 nearest anchors in Euclidean distance over the joint vector
// z_t = [k_t of all heads; v_t of all heads] (2 G d elements).
//
//   anc_norms    ||z_a||^2 of every anchor (fp32, fixed summation order)
//   anc_search   distance GEMM <z_a, z_t> by bf16 MFMA (the bf16 inputs are exact, the fp32
//                accumulation is the only rounding) on 128-anchor x 128-token tiles; ranking
//                key ||z_a||^2 - 2 <z_a, z_t> (||z_t||^2 is common to a token's candidates);
//                each tile leaves every token's 4 best (key, anchor) pairs
//   anc_merge    a token's partial lists -> its 4 nearest anchors, nearest first (ties to the
//                lower anchor number)
//   anc_prep     coded salience gathered from the prefix's, residuals k_t - mean, v_t - mean
//                (fp32, stored in the layer's dtype) followed by the window rows, and the
//                anchor rows copied to their store
//   anc_lists    after the allocation: the anchors of each stored position, per anchor the
//                stored positions that use it (counts, scan, fill), and those lists cut into
//                pieces of 64 entries (hub anchors are used by most tokens)
#include "vr_internal.h"

namespace vr {

constexpr int AN_C = 4;                 // nearest anchors per coded token
constexpr int AN_TT = 128;              // tokens per search tile
constexpr int AN_TA = 128;              // anchors per search tile

__host__ __device__ inline int64_t anc_token(int64_t i, int delta) { return i + i / (delta - 1) + 1; }

// ---- anchor norms: one wave per anchor
__global__ __launch_bounds__(256) void anc_norms(const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
                                                int64_t na, int delta, int GD, float* __restrict__ nrm) {
    const int64_t a = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (a >= na) return;
    const int64_t t = a * delta;
    float s = 0.f;
    for (int k = lane; k < 2 * GD; k += 64) {
        const float x = bf16_to_f32(k < GD ? K[t * GD + k] : V[t * GD + k - GD]);
        s = fmaf(x, x, s);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0) nrm[a] = s;
}

// Running 4 best (smallest key, ties to the smaller anchor number), sorted.
struct Top4 {
    float k[AN_C];
    uint32_t a[AN_C];
};
__device__ __forceinline__ bool anc_less(float k1, uint32_t a1, float k2, uint32_t a2) {
    return k1 < k2 || (k1 == k2 && a1 < a2);
}
__device__ __forceinline__ void top4_init(Top4& t) {
#pragma unroll
    for (int j = 0; j < AN_C; ++j) { t.k[j] = INFINITY; t.a[j] = 0xFFFFFFFFu; }
}
__device__ __forceinline__ void top4_push(Top4& t, float k, uint32_t a) {
    if (!anc_less(k, a, t.k[AN_C - 1], t.a[AN_C - 1])) return;
    t.k[AN_C - 1] = k;
    t.a[AN_C - 1] = a;
#pragma unroll
    for (int j = AN_C - 1; j > 0; --j) {
        if (anc_less(t.k[j], t.a[j], t.k[j - 1], t.a[j - 1])) {
            const float tk = t.k[j]; t.k[j] = t.k[j - 1]; t.k[j - 1] = tk;
            const uint32_t ta = t.a[j]; t.a[j] = t.a[j - 1]; t.a[j - 1] = ta;
        }
    }
}

// ---- distance GEMM + per-tile top 4.  Workgroup: 4 waves, 128 anchors x 128 tokens; wave
// (wa, wt) = (wave / 2, wave % 2) computes anchors 64 wa .. 64 wa + 63 (four 16-row tiles, A
// operand) against tokens 64 wt .. 64 wt + 63 (four 16-column tiles, B operand): 16 MFMA
// 16x16x32 per step of 32 elements of z.  Both operands are staged in LDS in fragment order by
// direct-to-LDS loads: one 1 KB load per 16-row (or 16-column) tile and step, lane l bringing
// row l % 16's elements 8 (l / 16) .. + 7, so every fragment read is one conflict-free 16-byte
// read per lane.  AS_NS stages of 16 KB rotate (each wave issues 4 loads per stage and waits
// on its own load count); a step's barrier also frees the buffer the next issue reuses.  Three
// stages measured best: 0.53 ms for the 32K layer against 0.61 with four and 0.82 with eight
// (one workgroup per CU then), and 0.65 ms for the earlier form (one step of lookahead, the
// token operand loaded straight into registers).
// C[anchor][token]: lane -> token column (lane % 16) and anchors 4 (lane / 16) + v of each
// 16-anchor row tile.  Workgroups are mapped so that all anchor tiles of one token tile run on
// the same XCD (its token rows stay in that XCD's L2).
constexpr int AS_NS = 3;                                 // stages in the ring (three workgroups per CU)
constexpr int AS_STAGE = (AN_TA / 16 + AN_TT / 16) * 1024;   // bytes per stage (A then B tiles)
constexpr size_t AS_LDS = (size_t)AS_NS * AS_STAGE;      // 48 KB
static_assert(AN_TA == 128 && AN_TT == 128, "one 1 KB load per 16-row tile; 16 loads per stage");

struct AnSearch {
    const uint16_t* K;
    const uint16_t* V;
    const float* nrm;
    float* pk;          // [n_atiles][Nc][4] partial keys
    uint32_t* pa;       // [n_atiles][Nc][4] partial anchor numbers
    int64_t Nc, na;
    int delta, GD, n_ttiles, n_atiles;
};

__device__ __forceinline__ const uint16_t* anc_zrow(const AnSearch& p, int64_t t, int k) {
    // element k (a multiple of 8) of z_t
    return k < p.GD ? p.K + t * p.GD + k : p.V + t * p.GD + (k - p.GD);
}

__global__ __launch_bounds__(256) void anc_search(AnSearch p) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int col = lane & 15, grp = lane >> 4;
    const int wa = wave >> 1, wt = wave & 1;
    // XCD-aware order: the 8 XCDs take consecutive workgroup ids in turn
    const int b = blockIdx.x;
    const int xcd = b & 7, k = b >> 3;
    const int tt = xcd + 8 * (k / p.n_atiles), at = k % p.n_atiles;
    if (tt >= p.n_ttiles) return;
    const int64_t i0 = (int64_t)tt * AN_TT;
    const int64_t a0 = (int64_t)at * AN_TA;
    // this wave's loads of a stage: A row tiles 2 wave, 2 wave + 1 and B column tiles 2 wave,
    // 2 wave + 1; lane row l % 16, elements 8 (l / 16) .. + 7 of the step (rows clamped: rows
    // past the anchors or tokens are dropped later)
    int64_t lrow[4];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        int64_t a = a0 + 16 * (2 * wave + u) + col;
        a = a < p.na ? a : p.na - 1;
        lrow[u] = a * p.delta;
        int64_t i = i0 + 16 * (2 * wave + u) + col;
        i = i < p.Nc ? i : p.Nc - 1;
        lrow[2 + u] = anc_token(i, p.delta);
    }
    const uint32_t lds0 = __builtin_amdgcn_readfirstlane((uint32_t)(size_t)(__attribute__((address_space(3))) uint8_t*)smem);
    const int steps = 2 * p.GD / 32;
    auto issue = [&](int s) {
        const int kk = 32 * s + 8 * grp;
        const uint32_t st = lds0 + (uint32_t)(s % AS_NS) * AS_STAGE;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            // tile index in the stage: A tiles 0..7, then B tiles 8..15
            const uint32_t dst = st + 1024u * (uint32_t)((u < 2 ? 0 : 8) + 2 * wave + (u & 1));
            asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                         :: "v"(anc_zrow(p, lrow[u], kk)), "s"(dst) : "memory", "m0");
        }
    };
    f32x4 acc[4][4];                          // [row tile][column tile] of this wave
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[j][c] = f32x4{0, 0, 0, 0};
    for (int s = 0; s < AS_NS - 1 && s < steps; ++s) issue(s);
    for (int s = 0; s < steps; ++s) {
        // stage s has landed when at most the loads of the stages after it are in flight
        static_assert(AS_NS == 3, "the wait below leaves one later stage (4 loads) in flight");
        if (s + AS_NS - 2 < steps) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
        else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();                      // every wave's part of stage s; stage s - 1 is free
        if (s + AS_NS - 1 < steps) issue(s + AS_NS - 1);
        const u32x4* sa = reinterpret_cast<const u32x4*>(smem + (size_t)(s % AS_NS) * AS_STAGE);
        const u32x4* sb = sa + 8 * 64;
        u32x4 fa[4], fb[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) fa[j] = sa[(4 * wa + j) * 64 + lane];
#pragma unroll
        for (int c = 0; c < 4; ++c) fb[c] = sb[(4 * wt + c) * 64 + lane];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int c = 0; c < 4; ++c) acc[j][c] = mfma(fa[j], fb[c], acc[j][c]);
    }
    // ---- keys and the 4 best per token of this wave's 64 anchors: per lane, then over the 4
    //      lanes of a token; then the two anchor halves of the workgroup through LDS
    __syncthreads();                          // every wave is done with the stages
    float* xk = reinterpret_cast<float*>(smem);                  // [wt][4 col tiles][16][4]
    uint32_t* xa = reinterpret_cast<uint32_t*>(smem + 2 * 4 * 16 * AN_C * 4);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        Top4 t;
        top4_init(t);
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t a = a0 + 64 * wa + 16 * j + 4 * grp + v;
                if (a < p.na) top4_push(t, p.nrm[a] - 2.f * acc[j][c][v], (uint32_t)a);
            }
#pragma unroll
        for (int m = 16; m <= 32; m <<= 1) {
            float ok[AN_C];
            uint32_t oa[AN_C];
#pragma unroll
            for (int q = 0; q < AN_C; ++q) {
                ok[q] = __shfl_xor(t.k[q], m, 64);
                oa[q] = (uint32_t)__shfl_xor((int)t.a[q], m, 64);
            }
#pragma unroll
            for (int q = 0; q < AN_C; ++q) top4_push(t, ok[q], oa[q]);
        }
        const int slot = ((wt * 4 + c) * 16 + col) * AN_C;
        if (wa == 1 && grp == 0) {
#pragma unroll
            for (int q = 0; q < AN_C; ++q) { xk[slot + q] = t.k[q]; xa[slot + q] = t.a[q]; }
        }
        __syncthreads();
        if (wa == 0) {
#pragma unroll
            for (int q = 0; q < AN_C; ++q) top4_push(t, xk[slot + q], xa[slot + q]);
            const int64_t i = i0 + 64 * wt + 16 * c + col;
            if (grp == 0 && i < p.Nc) {
                const int64_t o = ((int64_t)at * p.Nc + i) * AN_C;
#pragma unroll
                for (int q = 0; q < AN_C; ++q) { p.pk[o + q] = t.k[q]; p.pa[o + q] = t.a[q]; }
            }
        }
    }
}

// ---- merge of the partial lists: one thread per coded token
__global__ __launch_bounds__(256) void anc_merge(const float* __restrict__ pk, const uint32_t* __restrict__ pa,
                                                int64_t Nc, int n_atiles, uint16_t* __restrict__ nn) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= Nc) return;
    Top4 t;
    top4_init(t);
    for (int at = 0; at < n_atiles; ++at) {
        const int64_t o = ((int64_t)at * Nc + i) * AN_C;
#pragma unroll
        for (int q = 0; q < AN_C; ++q) top4_push(t, pk[o + q], pa[o + q]);
    }
#pragma unroll
    for (int q = 0; q < AN_C; ++q) nn[i * AN_C + q] = (uint16_t)t.a[q];
}

// ---- compaction, residuals and the anchor store.  One wave per (row, head) piece of 128
// elements; rows: coded tokens i < Nc (residual), window rows (copied), anchors (copied).
template <typename ET>
__global__ __launch_bounds__(256) void anc_prep(const ET* __restrict__ K, const ET* __restrict__ V,
                                               const float* __restrict__ sbar, const uint16_t* __restrict__ nn,
                                               int64_t N, int64_t Nc, int64_t na, int w, int G, int delta,
                                               float* __restrict__ sbar_c, ET* __restrict__ Kr, ET* __restrict__ Vr,
                                               ET* __restrict__ Ka, ET* __restrict__ Va) {
    const int64_t piece = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int64_t rows = Nc + w + na;
    if (piece >= rows * G) return;
    const int64_t r = piece / G;
    const int g = (int)(piece % G);
    const int GD = G * D;
    for (int e = lane; e < D; e += 64) {
        if (r < Nc) {
            const int64_t t = anc_token(r, delta);
            float mk = 0.f, mv = 0.f;
#pragma unroll
            for (int q = 0; q < AN_C; ++q) {            // fixed order: nearest first
                const int64_t ta = (int64_t)nn[r * AN_C + q] * delta;
                mk += elem_f(K[ta * GD + g * D + e]);
                mv += elem_f(V[ta * GD + g * D + e]);
            }
            mk *= 1.f / AN_C;
            mv *= 1.f / AN_C;
            Kr[r * GD + g * D + e] = to_elem<ET>(elem_f(K[t * GD + g * D + e]) - mk);
            Vr[r * GD + g * D + e] = to_elem<ET>(elem_f(V[t * GD + g * D + e]) - mv);
            if (g == 0 && e == 0) sbar_c[r] = sbar[t];
        } else if (r < Nc + w) {
            const int64_t t = N + (r - Nc);
            Kr[r * GD + g * D + e] = K[t * GD + g * D + e];
            Vr[r * GD + g * D + e] = V[t * GD + g * D + e];
        } else {
            const int64_t a = r - Nc - w;
            Ka[a * GD + g * D + e] = K[a * delta * GD + g * D + e];
            Va[a * GD + g * D + e] = V[a * delta * GD + g * D + e];
        }
    }
}

// ---- after the allocation: anchors of every stored position, and the inverse lists
__global__ __launch_bounds__(256) void anc_count(const uint32_t* __restrict__ sidx, const uint16_t* __restrict__ nn,
                                                int64_t Nc, uint16_t* __restrict__ snn, uint32_t* __restrict__ cnt) {
    const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (p >= Nc) return;
    const int64_t i = sidx[p];
#pragma unroll
    for (int q = 0; q < AN_C; ++q) {
        const uint16_t a = nn[i * AN_C + q];
        snn[p * AN_C + q] = a;
        atomicAdd(&cnt[a], 1u);
    }
}

// exclusive scan of na counts (one workgroup); the counts become fill cursors (set to the
// list starts)
__global__ __launch_bounds__(1024) void anc_scan(uint32_t* __restrict__ cnt, int64_t na, uint32_t* __restrict__ off) {
    __shared__ uint32_t part[1024];
    const int tid = threadIdx.x;
    const int64_t per = (na + 1023) / 1024;
    const int64_t b0 = tid * per;
    uint32_t s = 0;
    for (int64_t a = b0; a < b0 + per && a < na; ++a) s += cnt[a];
    part[tid] = s;
    __syncthreads();
    for (int o = 1; o < 1024; o <<= 1) {
        const uint32_t v = tid >= o ? part[tid - o] : 0u;
        __syncthreads();
        part[tid] += v;
        __syncthreads();
    }
    uint32_t run = tid ? part[tid - 1] : 0u;
    for (int64_t a = b0; a < b0 + per && a < na; ++a) {
        const uint32_t c = cnt[a];
        off[a] = run;
        cnt[a] = run;
        run += c;
    }
    if (tid == 1023) off[na] = part[1023];
}

__global__ __launch_bounds__(256) void anc_fill(const uint16_t* __restrict__ snn, int64_t Nc,
                                               uint32_t* __restrict__ cur, uint32_t* __restrict__ inv) {
    const int64_t p = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (p >= Nc) return;
#pragma unroll
    for (int q = 0; q < AN_C; ++q) {
        const uint32_t slot = atomicAdd(&cur[snn[p * AN_C + q]], 1u);
        inv[slot] = (uint32_t)p;
    }
}

// pieces of 64 entries per anchor list (hub anchors, used by a large share of the tokens,
// have long lists): counts, then (after a scan into piece_off) each piece's anchor
__global__ __launch_bounds__(256) void anc_pcount(const uint32_t* __restrict__ off, int64_t na, uint32_t* __restrict__ cnt) {
    const int64_t a = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (a < na) cnt[a] = (off[a + 1] - off[a] + 63) / 64;
}
__global__ __launch_bounds__(256) void anc_pfill(const uint32_t* __restrict__ poff, int64_t na,
                                                uint16_t* __restrict__ panchor) {
    const int64_t a = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (a >= na) return;
    for (uint32_t k = poff[a]; k < poff[a + 1]; ++k) panchor[k] = (uint16_t)a;
}

__global__ void anc_zero(uint32_t* __restrict__ x, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) x[i] = 0u;
}

// ----------------------------------------------------------------------------------------
static inline int anc_atiles(const varrate_shape& sh) { return (int)((anchor_count(sh) + AN_TA - 1) / AN_TA); }

size_t anchor_ws_bytes(const varrate_shape& sh) {
    const int64_t Np = sh.n - sh.w, Nc = coded_count(sh), na = anchor_count(sh);
    const size_t rows = (size_t)(Nc + sh.w) * sh.G * D * 2;
    return align256(salience_ws_bytes(sh)) + align256(allocate_ws_bytes(sh)) + align256((size_t)Np * 4) +
           align256((size_t)Nc * 4) + align256((size_t)na * 4) + 2 * align256((size_t)anc_atiles(sh) * Nc * AN_C * 4) +
           align256((size_t)Nc * AN_C * 2) + 2 * align256(rows) + align256((size_t)na * 4);
}

AnchorWs anchor_ws(const varrate_shape& sh, uint8_t* ws) {
    const int64_t Np = sh.n - sh.w, Nc = coded_count(sh), na = anchor_count(sh);
    const size_t rows = (size_t)(Nc + sh.w) * sh.G * D * 2;
    AnchorWs w;
    uint8_t* p = ws;
    w.sal = p;                p += align256(salience_ws_bytes(sh));
    w.alloc = p;              p += align256(allocate_ws_bytes(sh));
    w.sbar = (float*)p;       p += align256((size_t)Np * 4);
    w.sbar_c = (float*)p;     p += align256((size_t)Nc * 4);
    w.nrm = (float*)p;        p += align256((size_t)na * 4);
    w.pk = (float*)p;         p += align256((size_t)anc_atiles(sh) * Nc * AN_C * 4);
    w.pa = (uint32_t*)p;      p += align256((size_t)anc_atiles(sh) * Nc * AN_C * 4);
    w.nn = (uint16_t*)p;      p += align256((size_t)Nc * AN_C * 2);
    w.Kr = p;                 p += align256(rows);
    w.Vr = p;                 p += align256(rows);
    w.cnt = (uint32_t*)p;
    return w;
}

hipError_t launch_anchor_search(const varrate_shape& sh, const void* K, const void* V, uint16_t* nn,
                                const AnchorWs& w, hipStream_t st) {
    const int64_t Nc = coded_count(sh), na = anchor_count(sh);
    const int GD = sh.G * D;
    anc_norms<<<(unsigned)((na + 3) / 4), 256, 0, st>>>((const uint16_t*)K, (const uint16_t*)V, na,
                                                        sh.anchor_stride, GD, w.nrm);
    AnSearch p;
    p.K = (const uint16_t*)K;
    p.V = (const uint16_t*)V;
    p.nrm = w.nrm;
    p.pk = w.pk;
    p.pa = w.pa;
    p.Nc = Nc;
    p.na = na;
    p.delta = sh.anchor_stride;
    p.GD = GD;
    p.n_ttiles = (int)((Nc + AN_TT - 1) / AN_TT);
    p.n_atiles = anc_atiles(sh);
    // 8 XCDs, each with ceil(n_ttiles / 8) token tiles x n_atiles anchor tiles
    const int64_t per_xcd = (int64_t)((p.n_ttiles + 7) / 8) * p.n_atiles;
    hipError_t e = ensure_lds_limit((const void*)anc_search, AS_LDS);
    if (e != hipSuccess) return e;
    anc_search<<<(unsigned)(8 * per_xcd), 256, AS_LDS, st>>>(p);
    anc_merge<<<(unsigned)((Nc + 255) / 256), 256, 0, st>>>(w.pk, w.pa, Nc, p.n_atiles, nn);
    return hipGetLastError();
}

hipError_t launch_anchor_encode(const varrate_shape& sh, const void* K, const void* V, const float* sbar,
                                const uint16_t* nn, const float* PK, const float* PV, varrate_cache& c,
                                const AnchorWs& w, hipStream_t st) {
    const int64_t Np = sh.n - sh.w, Nc = coded_count(sh), na = anchor_count(sh);
    const varrate_shape shc = coded_shape(sh);
    const int64_t pieces = (Nc + sh.w + na) * sh.G;
    anc_prep<uint16_t><<<(unsigned)((pieces + 3) / 4), 256, 0, st>>>(
        (const uint16_t*)K, (const uint16_t*)V, sbar, nn, Np, Nc, na, sh.w, sh.G, sh.anchor_stride, w.sbar_c,
        (uint16_t*)w.Kr, (uint16_t*)w.Vr, (uint16_t*)c.k_anchor, (uint16_t*)c.v_anchor);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const uint32_t* csz = nullptr;
    if ((e = launch_allocate(shc, w.sbar_c, c, w.alloc, st, nullptr, &csz)) != hipSuccess) return e;
    if ((e = launch_project(shc, w.Kr, w.Vr, PK, PV, c, st, csz)) != hipSuccess) return e;
    anc_zero<<<(unsigned)((na + 255) / 256), 256, 0, st>>>(w.cnt, na);
    anc_count<<<(unsigned)((Nc + 255) / 256), 256, 0, st>>>(c.sidx, nn, Nc, c.snn, w.cnt);
    anc_scan<<<1, 1024, 0, st>>>(w.cnt, na, c.inv_off);
    anc_fill<<<(unsigned)((Nc + 255) / 256), 256, 0, st>>>(c.snn, Nc, w.cnt, c.inv_pos);
    anc_pcount<<<(unsigned)((na + 255) / 256), 256, 0, st>>>(c.inv_off, na, w.cnt);
    anc_scan<<<1, 1024, 0, st>>>(w.cnt, na, c.piece_off);
    anc_pfill<<<(unsigned)((na + 255) / 256), 256, 0, st>>>(c.piece_off, na, c.piece_anchor);
    return hipGetLastError();
}

}  // namespace vr
