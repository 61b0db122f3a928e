// Basis projection + nested truncation + packing (Sec. 3.3 Eq. (6), Algorithm 1), gfx950.
//
// One workgroup per (group of PJ_CPW chunks, KV head g, K|V), two workgroups per CU.
//   1. Storage order.  Each chunk's tokens are put in (rank descending, index ascending)
//      order by a stable counting sort: every token sets its bit in a per-rank 256-bit
//      mask, a token's position is (#tokens of higher rank) + (#lower-index tokens of its
//      rank), both read off the masks with popcounts.  The (head 0, K) workgroup publishes
//      srank / sidx.
//   2. The basis P (fp32) is split into bf16 hi + lo parts once per workgroup and kept in
//      LDS in MFMA-fragment order (64 KB), so every product is P_hi x + P_lo x with exact
//      bf16 x (fp32 x adds P_hi x_lo): about 2^-16 relative error before storage rounding.
//   3. Waves take 32-token super-tiles; a super-tile only computes the 16-row coefficient
//      blocks j below its largest rank (its first token's).  Token fragments of the next
//      super-tile are loaded while the current one is multiplied (a fixed number of loads,
//      so the wait counts stay exact).  The C tile (16 coefficients x 16 tokens) goes
//      straight into the ragged packed rows.
// Workgroups of chunk group 0 also copy the window rows into the exact slots.
#include "vr_internal.h"

namespace vr {

constexpr int PJ_THREADS = 512;     // 8 waves
constexpr int PJ_CPW = 4;           // chunks per workgroup
constexpr int PJ_FRAGS = 8 * 4;     // (16-row block a, 32-col step s) pairs
constexpr int NR = D + 1;           // rank values 0..128

struct PjSmem {
    u32x4* frag_hi;                 // [32][64]
    u32x4* frag_lo;                 // [32][64]
    unsigned long long* mask;       // [2][NR][4] rank masks of two chunks being sorted
    uint16_t* s_tok;                // [CPW][256] local token index of stored slot
    uint16_t* s_off;                // [CPW][256] local coefficient offset
    uint8_t* s_rank;                // [CPW][256]
    uint16_t* start;                // [2][NR]
};

static inline size_t project_smem_bytes() {
    return (size_t)PJ_FRAGS * 64 * 16 * 2 + (size_t)2 * NR * 4 * 8 + (size_t)PJ_CPW * CHUNK * 5 +
           (size_t)2 * NR * 2 + 16;
}

__device__ __forceinline__ PjSmem pj_carve(uint8_t* smem) {
    PjSmem s;
    s.frag_hi = reinterpret_cast<u32x4*>(smem);
    s.frag_lo = s.frag_hi + PJ_FRAGS * 64;
    s.mask = reinterpret_cast<unsigned long long*>(s.frag_lo + PJ_FRAGS * 64);
    s.s_tok = reinterpret_cast<uint16_t*>(s.mask + 2 * NR * 4);
    s.s_off = s.s_tok + PJ_CPW * CHUNK;
    s.s_rank = reinterpret_cast<uint8_t*>(s.s_off + PJ_CPW * CHUNK);
    s.start = reinterpret_cast<uint16_t*>(s.s_rank + PJ_CPW * CHUNK);
    return s;
}

template <bool F32>
struct XFrag {
    u32x4 h[2][4];
    u32x4 l[2][4];
};

template <bool F32>
__device__ __forceinline__ void load_x(XFrag<F32>& xf, const void* X, const PjSmem& sm, int cc, int i0,
                                       int T, int64_t t0, int G, int g, int grp, int col) {
#pragma unroll
    for (int hb = 0; hb < 2; ++hb) {
        const int i = i0 + 16 * hb + col;
        // slots past the chunk's end read token t0 (valid memory); their columns are never stored
        const int64_t t = t0 + (i < T ? sm.s_tok[cc * CHUNK + i] : 0);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int64_t e0 = (t * G + g) * D + 32 * s + 8 * grp;
            if constexpr (!F32) {
                xf.h[hb][s] = load16((const uint16_t*)X + e0);
            } else {
                xf.h[hb][s] = load16((const float*)X + e0);
                xf.l[hb][s] = load16((const float*)X + e0 + 4);
            }
        }
    }
}

template <bool F32>
__global__ __launch_bounds__(PJ_THREADS, F32 ? 2 : 4) void project_kernel(
    const void* __restrict__ K, const void* __restrict__ V, const float* __restrict__ PK,
    const float* __restrict__ PV, int64_t N, int G, int w, const uint8_t* __restrict__ rank,
    uint8_t* __restrict__ srank, uint32_t* __restrict__ sidx, const uint32_t* __restrict__ chunk_off,
    int n_chunks, void* __restrict__ coef_k, void* __restrict__ coef_v, int64_t coef_stride,
    void* __restrict__ k_exact, void* __restrict__ v_exact, int64_t cap) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    PjSmem sm = pj_carve(smem);
    __shared__ uint32_t s_base[PJ_CPW];
    __shared__ int s_T[PJ_CPW];
    __shared__ int s_tiles[PJ_CPW + 1];

    const int g = blockIdx.y, kv = blockIdx.z;
    const void* X = kv ? V : K;
    const float* P = (kv ? PV : PK) + (int64_t)g * D * D;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int grp = lane >> 4, col = lane & 15;
    const int c0 = blockIdx.x * PJ_CPW;
    const bool publish = g == 0 && kv == 0;

    // ---- ranks of the 4 chunks (16-byte loads; the rank buffer is padded to 64)
    {
        if (tid < PJ_CPW) {
            const int c = c0 + tid;
            const int64_t t0 = (int64_t)c * CHUNK;
            s_T[tid] = c < n_chunks ? (int)((N - t0) < CHUNK ? (N - t0) : CHUNK) : 0;
            s_base[tid] = c < n_chunks ? chunk_off[c] : 0;
        }
        if (tid < PJ_CPW * CHUNK / 16) {
            const int64_t t = (int64_t)c0 * CHUNK + tid * 16;
            u32x4 v = {0, 0, 0, 0};
            if (t < N) v = load16(rank + t);
            // stage the original-order ranks in s_off's bytes until they are sorted
            *reinterpret_cast<u32x4*>(reinterpret_cast<uint8_t*>(sm.s_off) + tid * 16) = v;
        }
    }
    // ---- basis fragments: fragment f = a * 4 + s, lane l -> row 16a + l%16, cols 32s + 8(l/16)
    for (int idx = tid; idx < PJ_FRAGS * 64; idx += PJ_THREADS) {
        const int f = idx >> 6, l = idx & 63;
        const int a = f >> 2, s = f & 3;
        const float* src = P + (16 * a + (l & 15)) * D + 32 * s + 8 * (l >> 4);
        float x[8];
        u32x4 p0 = load16(src), p1 = load16(src + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) { x[e] = __uint_as_float(p0[e]); x[4 + e] = __uint_as_float(p1[e]); }
        split8(x, sm.frag_hi[idx], sm.frag_lo[idx]);
    }
    __syncthreads();
    const uint8_t* orig_rank = reinterpret_cast<const uint8_t*>(sm.s_off);
    // ---- stable counting sort of two chunks at a time (threads 0..255 / 256..511)
    for (int pass = 0; pass < PJ_CPW / 2; ++pass) {
        const int half = tid >> 8, i = tid & 255;
        const int cc = 2 * pass + half;
        unsigned long long* mk = sm.mask + half * NR * 4;
        for (int k = i; k < NR * 4; k += 256) mk[k] = 0ull;
        __syncthreads();
        const int T = s_T[cc];
        const int r = i < T ? orig_rank[cc * CHUNK + i] : -1;
        if (r >= 0) atomicOr(&mk[r * 4 + (i >> 6)], 1ull << (i & 63));
        __syncthreads();
        // start[r] = tokens of rank > r: the first wave of each half scans ranks 128..0
        if ((tid & 255) < 64) {
            const int ln = tid & 63;
            uint32_t h[3], loc = 0;
#pragma unroll
            for (int e = 0; e < 3; ++e) {
                const int k = 3 * ln + e;       // descending slot k <-> rank 128 - k
                h[e] = 0;
                if (k < NR) {
                    const unsigned long long* m = mk + (NR - 1 - k) * 4;
                    h[e] = __popcll(m[0]) + __popcll(m[1]) + __popcll(m[2]) + __popcll(m[3]);
                }
                loc += h[e];
            }
            uint32_t xs = loc;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                uint32_t y = __shfl_up(xs, off, 64);
                if (ln >= off) xs += y;
            }
            uint32_t pre = xs - loc;
#pragma unroll
            for (int e = 0; e < 3; ++e) {
                const int k = 3 * ln + e;
                if (k < NR) sm.start[half * NR + (NR - 1 - k)] = (uint16_t)pre;
                pre += h[e];
            }
        }
        __syncthreads();
        if (r >= 0) {
            const unsigned long long* m = mk + r * 4;
            uint32_t below = 0;
            const int wd = i >> 6;
#pragma unroll
            for (int k = 0; k < 4; ++k)
                if (k < wd) below += __popcll(m[k]);
            below += __popcll(m[wd] & ((1ull << (i & 63)) - 1ull));
            const int pos = sm.start[half * NR + r] + below;
            sm.s_tok[cc * CHUNK + pos] = (uint16_t)i;
            sm.s_rank[cc * CHUNK + pos] = (uint8_t)r;
            if (publish) {
                const int64_t t0 = (int64_t)(c0 + cc) * CHUNK;
                srank[t0 + pos] = (uint8_t)r;
                sidx[t0 + pos] = (uint32_t)(t0 + i);
            }
        }
        __syncthreads();
    }
    // ---- local offsets: wave cc scans chunk cc (4 entries per lane)
    if (wave < PJ_CPW) {
        const int cc = wave;
        const int T = s_T[cc];
        uint32_t r[4], loc = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) { r[e] = 4 * lane + e < T ? sm.s_rank[cc * CHUNK + 4 * lane + e] : 0; loc += r[e]; }
        uint32_t x = loc;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            uint32_t y = __shfl_up(x, off, 64);
            if (lane >= off) x += y;
        }
        uint32_t pre = x - loc;
#pragma unroll
        for (int e = 0; e < 4; ++e) { sm.s_off[cc * CHUNK + 4 * lane + e] = (uint16_t)pre; pre += r[e]; }
    }
    if (tid == 0) {
        int acc = 0;
        for (int cc = 0; cc < PJ_CPW; ++cc) { s_tiles[cc] = acc; acc += (s_T[cc] + 31) / 32; }
        s_tiles[PJ_CPW] = acc;
    }
    __syncthreads();

    // ---- projection of 32-token super-tiles, next super-tile's fragments in flight
    const int ntiles = s_tiles[PJ_CPW];
    auto locate = [&](int tile, int& cc, int& i0) {
        cc = 0;
        while (tile >= s_tiles[cc + 1]) ++cc;
        i0 = (tile - s_tiles[cc]) * 32;
    };
    if (wave < ntiles) {
        XFrag<F32> cur, nxt;
        int cc, i0;
        locate(wave, cc, i0);
        load_x<F32>(cur, X, sm, cc, i0, s_T[cc], (int64_t)(c0 + cc) * CHUNK, G, g, grp, col);
        for (int tile = wave; tile < ntiles; tile += PJ_THREADS / 64) {
            const int nt = tile + PJ_THREADS / 64 < ntiles ? tile + PJ_THREADS / 64 : tile;
            int ncc, ni0;
            locate(nt, ncc, ni0);
            load_x<F32>(nxt, X, sm, ncc, ni0, s_T[ncc], (int64_t)(c0 + ncc) * CHUNK, G, g, grp, col);
            const int T = s_T[cc];
            const int rmax = sm.s_rank[cc * CHUNK + i0];
            const int na = rmax < D ? (rmax + 15) >> 4 : D / 16;
            u32x4 xh[2][4], xl[2][4];
#pragma unroll
            for (int hb = 0; hb < 2; ++hb)
#pragma unroll
                for (int s = 0; s < 4; ++s) {
                    if constexpr (!F32) {
                        xh[hb][s] = cur.h[hb][s];
                        xl[hb][s] = u32x4{0, 0, 0, 0};
                    } else {
                        float x8[8];
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            x8[e] = __uint_as_float(cur.h[hb][s][e]);
                            x8[4 + e] = __uint_as_float(cur.l[hb][s][e]);
                        }
                        split8(x8, xh[hb][s], xl[hb][s]);
                    }
                }
            int r_of[2], o_of[2];
#pragma unroll
            for (int hb = 0; hb < 2; ++hb) {
                const int i = i0 + 16 * hb + col;
                r_of[hb] = i < T ? sm.s_rank[cc * CHUNK + i] : 0;
                o_of[hb] = i < T ? sm.s_off[cc * CHUNK + i] : 0;
                // stores stay inside the head's stream whatever the layout tables hold
                const int64_t room = coef_stride - ((int64_t)s_base[cc] + o_of[hb]);
                r_of[hb] = room < r_of[hb] ? (room > 0 ? (int)room : 0) : r_of[hb];
            }
            const int64_t out0 = (int64_t)g * coef_stride + s_base[cc];
            for (int a = 0; a < na; ++a) {
                u32x4 ph[4], pl[4];
#pragma unroll
                for (int s = 0; s < 4; ++s) {
                    ph[s] = sm.frag_hi[(a * 4 + s) * 64 + lane];
                    pl[s] = sm.frag_lo[(a * 4 + s) * 64 + lane];
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
                    // C: lane -> token column (slot i0 + 16hb + col), rows j0 .. j0 + 3 with
                    // j0 = 16a + 4grp: four consecutive coefficients of one packed row, stored
                    // at once unless the row ends inside them
                    const int r = r_of[hb];
                    const int j0 = 16 * a + 4 * grp;
                    const int64_t dst = out0 + o_of[hb] + j0;
                    if constexpr (F32) {
                        float* o = (float*)(kv ? coef_v : coef_k) + dst;
                        if (j0 + 4 <= r) {
                            __builtin_memcpy(o, &c, 16);
                        } else {
#pragma unroll
                            for (int v = 0; v < 3; ++v)
                                if (j0 + v < r) o[v] = c[v];
                        }
                    } else {
                        uint16_t* o = (uint16_t*)(kv ? coef_v : coef_k) + dst;
                        const uint32_t p01 = cvt_bf16x2(c[0], c[1]), p23 = cvt_bf16x2(c[2], c[3]);
                        if (j0 + 4 <= r) {
                            const uint2 pk = make_uint2(p01, p23);
                            __builtin_memcpy(o, &pk, 8);
                        } else {
                            if (j0 < r) o[0] = (uint16_t)p01;
                            if (j0 + 1 < r) o[1] = (uint16_t)(p01 >> 16);
                            if (j0 + 2 < r) o[2] = (uint16_t)p23;
                        }
                    }
                }
            }
            cur = nxt;
            cc = ncc;
            i0 = ni0;
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

template <bool F32>
static hipError_t pj_attr(size_t bytes) {
    static size_t done = 0;
    if (bytes <= done) return hipSuccess;
    hipError_t e = hipFuncSetAttribute((const void*)project_kernel<F32>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e == hipSuccess) done = bytes;
    return e;
}

hipError_t launch_project(const varrate_shape& sh, const void* K, const void* V, const float* PK,
                          const float* PV, varrate_cache& c, hipStream_t st) {
    const int64_t N = sh.n - sh.w;
    const int n_chunks = (int)((N + CHUNK - 1) / CHUNK);
    dim3 grid((n_chunks + PJ_CPW - 1) / PJ_CPW, sh.G, 2);
    const size_t lds = project_smem_bytes();
    if (sh.dtype == VARRATE_BF16) {
        hipError_t e = pj_attr<false>(lds);
        if (e != hipSuccess) return e;
        project_kernel<false><<<grid, PJ_THREADS, lds, st>>>(
            K, V, PK, PV, N, sh.G, sh.w, c.rank, c.srank, c.sidx, c.chunk_off, n_chunks, c.coef_k,
            c.coef_v, c.coef_stride, c.k_exact, c.v_exact, c.cap);
    } else {
        hipError_t e = pj_attr<true>(lds);
        if (e != hipSuccess) return e;
        project_kernel<true><<<grid, PJ_THREADS, lds, st>>>(
            K, V, PK, PV, N, sh.G, sh.w, c.rank, c.srank, c.sidx, c.chunk_off, n_chunks, c.coef_k,
            c.coef_v, c.coef_stride, c.k_exact, c.v_exact, c.cap);
    }
    return hipGetLastError();
}

}  // namespace vr
