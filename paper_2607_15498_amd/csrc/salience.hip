// Observation-window salience (Sec. 3.2 Eq. (4)) and the length-5 moving average, gfx950.
//
// For KV head g the window queries of its H/G query heads form `rows` = (H/G) * w query
// rows (row rho = hh * w + i: query head g*(H/G)+hh, window query i at position n-w+i).
// Logits x = <q_rho, k_t> / sqrt(d) come from bf16 MFMA tiles (16 rows x 16 keys x 32 d);
// fp32 inputs are split into bf16 hi + lo parts (three products), keeping ~2^-16 accuracy.
//
//   pass 1 (sal_rowstats): per (row, key block) running max / sum of exp over the causal
//            range;
//   pass 2 (sal_colsum):   per row, the global max M and 1/L from the pass-1 partials (every
//            workgroup for its own head), then per coded key t, the sum over rows of
//            exp(x - M) / L (every window
//            query sees every coded key, so no mask), summed over the group's rows in a
//            fixed order -> s_part[g][t];
//   pool   (sal_pool):     s_t = sum_g s_part[g][t] / (w H) (fixed order), then the centred
//            length-5 moving average with zero padding, rounded to fp32.
//
// Both passes give each workgroup (8 waves) a contiguous run of 32 KB key blocks of one KV
// head, double-buffered in LDS: block b + 2 is requested with direct-to-LDS loads into the
// buffer block b has just vacated, while block b + 1 is computed.  Every wave takes one or
// two 16-row tiles of the window rows (its query fragments load once per workgroup).  A
// block sits in LDS in 16-byte pieces, XOR-swizzled inside each key row, so the 16 lanes
// that read the same piece of 16 consecutive keys hit 16 different bank groups.
#include "vr_internal.h"

namespace vr {

constexpr int SL_THREADS = 512;            // 8 waves
constexpr int SL_WAVES = 8;
constexpr int SL_STAGE = 32768;            // bytes of keys per block (one LDS buffer)
constexpr int SL_MAX_RT = 2;               // row tiles per wave (rows <= 8 * 16 * 2 = 256)
constexpr int SL_LPB = SL_STAGE / 1024 / SL_WAVES;   // direct-to-LDS loads per wave per block (4)
constexpr int SL_SLOTS = 512;              // workgroups per launch: two per CU
constexpr int SL_MERGE_REG = 16;           // pass-1 partials per thread loaded at once in pass 2

// Wait until at most `left` of this wave's memory loads are outstanding (vmcnt; the export
// and LDS counters are left alone).  Loads complete in order for this counter.
template <int left>
__device__ __forceinline__ void wait_vm() {
    static_assert(left >= 0 && left < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((left & 15) | (7 << 4) | (15 << 8) | ((left >> 4) << 14));
}

template <bool B> struct SlTag { static constexpr bool value = B; };

template <bool F32> __host__ __device__ constexpr int sl_keys() { return SL_STAGE / (D * (F32 ? 4 : 2)); }
template <bool F32> __host__ __device__ constexpr int sl_pieces() { return D * (F32 ? 4 : 2) / 16; }

// Issue the block's keys k0 .. k0 + KB - 1 of head g into the stage.  Slot s (16 bytes)
// holds piece (s % P) ^ (k % P) of key k = s / P; keys past n read key n - 1 (masked later).
template <bool F32>
__device__ __forceinline__ void sl_issue(uint8_t* stage, const void* K, int64_t n, int G, int g, int64_t k0) {
    constexpr int P = sl_pieces<F32>();
    constexpr int BLOCKS = SL_STAGE / 1024;             // 64 slots (1 KB) per load
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int lane = threadIdx.x & 63;
    const size_t row_bytes = (size_t)D * (F32 ? 4 : 2);
#pragma unroll
    for (int b = 0; b < BLOCKS / SL_WAVES; ++b) {
        const int m = wave + SL_WAVES * b;
        const int s = 64 * m + lane;
        const int k = s / P, piece = (s % P) ^ (k % P);
        int64_t t = k0 + k;
        t = t < n ? t : n - 1;
        const uint8_t* src = (const uint8_t*)K + ((size_t)t * G + g) * row_bytes + 16 * piece;
        const uint32_t dst = __builtin_amdgcn_readfirstlane(
            (uint32_t)(size_t)(__attribute__((address_space(3))) uint8_t*)(stage + 1024 * m));
        // issued in asm so the compiler does not add its own wait for all of these loads
        // before the first LDS read; the stage waits below (vmcnt + barrier) order them
        asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                     :: "v"(src), "s"(dst) : "memory", "m0");
    }
}

// Query fragments (A operand) for row tile rt: lane row = 16 rt + l%16, K group l/16.
template <bool F32>
__device__ __forceinline__ void sl_qfrag(const void* Qw, int H, int w, int hpg, int g, int rows,
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
            // rows past `rows` read row 0: their logits are never used (pass 1 writes only
            // real rows; pass 2 weighs them by 1/L = 0), and no mask waits for the load
            qh[s] = load16((const uint16_t*)Qw + base + c0);
            ql[s] = u32x4{0, 0, 0, 0};
        } else {
            const float* src = (const float*)Qw + base + c0;
            const u32x4 a = load16(src), b = load16(src + 4);
            float x[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                x[e] = ok ? __uint_as_float(a[e]) : 0.f;
                x[4 + e] = ok ? __uint_as_float(b[e]) : 0.f;
            }
            split8(x, qh[s], ql[s]);
        }
    }
}

// Logit tile: rows 16 rt.. (the fragments) x keys 16 kt.. of the stage (C lane col = key).
template <bool F32>
__device__ __forceinline__ f32x4 sl_logits(const uint8_t* stage, int kt, const u32x4 (&qh)[4],
                                           const u32x4 (&ql)[4]) {
    constexpr int P = sl_pieces<F32>();
    const int lane = threadIdx.x & 63;
    const int k = kt * 16 + (lane & 15), grp = lane >> 4;
    const uint8_t* row = stage + (size_t)k * P * 16;
    f32x4 c = {0, 0, 0, 0};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        if constexpr (!F32) {
            const int piece = 4 * s + grp;
            const u32x4 kh = *reinterpret_cast<const u32x4*>(row + 16 * (piece ^ (k % P)));
            c = mfma(qh[s], kh, c);
        } else {
            const int p0 = 2 * (4 * s + grp);
            const u32x4 a = *reinterpret_cast<const u32x4*>(row + 16 * (p0 ^ (k % P)));
            const u32x4 b = *reinterpret_cast<const u32x4*>(row + 16 * ((p0 + 1) ^ (k % P)));
            float x[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) { x[e] = __uint_as_float(a[e]); x[4 + e] = __uint_as_float(b[e]); }
            u32x4 kh, kl;
            split8(x, kh, kl);
            c = mfma(qh[s], kh, c);
            c = mfma(ql[s], kh, c);
            c = mfma(qh[s], kl, c);
        }
    }
    return c;
}

// ----------------------------------------------------------------------------------------
// Block pipeline shared by both passes: buffers 0/1 hold blocks b0, b0+1, ..; `step(b, buf)`
// computes block b from its buffer.
// sl_prime requests the first two blocks; sl_pipeline then runs the loop.
template <bool F32>
__device__ __forceinline__ void sl_prime(uint8_t* lds, const void* K, int64_t n, int G, int g, int b0, int b1) {
    constexpr int KB = sl_keys<F32>();
    sl_issue<F32>(lds, K, n, G, g, (int64_t)b0 * KB);
    if (b0 + 1 < b1) sl_issue<F32>(lds + SL_STAGE, K, n, G, g, (int64_t)(b0 + 1) * KB);
}
template <bool F32, class Step>
__device__ __forceinline__ void sl_pipeline(uint8_t* lds, const void* K, int64_t n, int G, int g,
                                            int b0, int b1, Step step) {
    constexpr int KB = sl_keys<F32>();
    for (int b = b0; b < b1; ++b) {
        uint8_t* buf = lds + ((b - b0) & 1) * SL_STAGE;
        if (b + 1 < b1) wait_vm<SL_LPB>();       // block b landed; block b + 1 may be in flight
        else wait_vm<0>();
        __syncthreads();
        step(b, buf);
        __syncthreads();                          // every wave is done with this buffer
        if (b + 2 < b1) sl_issue<F32>(buf, K, n, G, g, (int64_t)(b + 2) * KB);
    }
}

// pass 1: stats[(g * rows + rho) * nw + wgi] = (max, sum exp(x - max)) over the causal keys
// of the blocks [wgi * bpw, ..) of head g.  Grid (nw, G).
template <bool F32>
__global__ __launch_bounds__(SL_THREADS, 4) void sal_rowstats(const void* __restrict__ K,
                                                              const void* __restrict__ Qw,
                                                              int64_t n, int G, int H, int w,
                                                              float2* __restrict__ stats, int nw, int bpw) {
    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
    constexpr int KB = sl_keys<F32>();
    constexpr int TPB = KB / 16;                  // key tiles per block
    constexpr int TPS = TPB < 4 ? TPB : 4;        // key tiles per rescale
    const int wgi = blockIdx.x, g = blockIdx.y;
    const int hpg = H / G, rows = hpg * w, nrt = (rows + 15) / 16;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int lane = threadIdx.x & 63;
    const int64_t N = n - w;
    const int nblk = (int)((n + KB - 1) / KB);
    const int b0 = wgi * bpw, b1 = b0 + bpw < nblk ? b0 + bpw : nblk;

    u32x4 qh[SL_MAX_RT][4], ql[SL_MAX_RT][4];
#pragma unroll
    for (int j = 0; j < SL_MAX_RT; ++j) {
        const int rt = wave + SL_WAVES * j;
        if (rt < nrt) sl_qfrag<F32>(Qw, H, w, hpg, g, rows, rt, qh[j], ql[j]);
    }
    // last visible key of each of this lane's rows (n - w + i for window query i); rows past
    // `rows` see nothing
    int tlast[SL_MAX_RT][4];                       // n < 2^31 (checked by the library)
#pragma unroll
    for (int j = 0; j < SL_MAX_RT; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int rho = (wave + SL_WAVES * j) * 16 + (lane >> 4) * 4 + v;
            tlast[j][v] = rho < rows ? (int)N + rho % w : -1;
        }
    // The block loads are issued in asm, unseen by the compiler's wait bookkeeping: every
    // load it knows of must land before them, or its own waits would drain the pipeline.
    wait_vm<0>();

    const float sl2 = 0.08838834764831845f * 1.4426950408889634f;   // log2(e) / sqrt(128)
    // Per lane and row: running max m and sum l of exp2 over this lane's keys, in log2
    // units, rescaled once per TPS key tiles (no per-element branches).
    float m[SL_MAX_RT][4], l[SL_MAX_RT][4];
#pragma unroll
    for (int j = 0; j < SL_MAX_RT; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) { m[j][v] = -INFINITY; l[j][v] = 0.f; }

    auto tiles = [&](const uint8_t* buf, int64_t k0, int64_t kend, int tq0, auto masked) {
#pragma unroll
        for (int j = 0; j < SL_MAX_RT; ++j) {
            const int rt = wave + SL_WAVES * j;
            if (rt >= nrt) continue;
            float x[TPS][4];
#pragma unroll
            for (int q = 0; q < TPS; ++q) {
                const int kt = tq0 + q;
                const f32x4 c = sl_logits<F32>(buf, kt, qh[j], ql[j]);
#pragma unroll
                for (int v = 0; v < 4; ++v) x[q][v] = c[v] * sl2;
                if constexpr (decltype(masked)::value) {
                    const int t = (int)k0 + kt * 16 + (lane & 15);
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        if (!(t < (int)kend && t <= tlast[j][v])) x[q][v] = -INFINITY;
                }
            }
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float mx = m[j][v];
#pragma unroll
                for (int q = 0; q < TPS; ++q) mx = fmaxf(mx, x[q][v]);
                if constexpr (decltype(masked)::value) {
                    if (mx == -INFINITY) continue;            // nothing visible yet here
                }
                float sum = l[j][v] * __builtin_amdgcn_exp2f(m[j][v] - mx);
#pragma unroll
                for (int q = 0; q < TPS; ++q) sum += __builtin_amdgcn_exp2f(x[q][v] - mx);
                l[j][v] = sum;
                m[j][v] = mx;
            }
        }
    };
    sl_prime<F32>(lds, K, n, G, g, b0, b1);
    sl_pipeline<F32>(lds, K, n, G, g, b0, b1, [&](int b, const uint8_t* buf) {
        const int64_t k0 = (int64_t)b * KB;
        const int64_t kend = k0 + KB < n ? k0 + KB : n;
        // every key of a full block that ends before the window is visible to every row
        if (kend - k0 == KB && kend <= N) {
#pragma unroll
            for (int tq = 0; tq < TPB; tq += TPS) tiles(buf, k0, kend, tq, SlTag<false>{});
        } else {
#pragma unroll
            for (int tq = 0; tq < TPB; tq += TPS) tiles(buf, k0, kend, tq, SlTag<true>{});
        }
    });

#pragma unroll
    for (int j = 0; j < SL_MAX_RT; ++j) {
        const int rt = wave + SL_WAVES * j;
        if (rt >= nrt) continue;
        // combine the 16 lanes (keys) that share a row (lane bits 0..3), in natural-log units:
        // the row's maximum over the lanes, then each lane's sum rescaled to it once and the
        // sums added over the lanes
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float mm = m[j][v] * 0.6931471805599453f;
            const float M = wave_max16(mm);
            float ll = mm == -INFINITY ? 0.f : l[j][v] * fast_exp(mm - M);
#pragma unroll
            for (int off = 1; off < 16; off <<= 1) ll += shfl_xor_f(ll, off);
            const int rho = rt * 16 + (lane >> 4) * 4 + v;
            if ((lane & 15) == 0 && rho < rows)
                stats[((int64_t)g * rows + rho) * nw + wgi] = make_float2(M, ll);
        }
    }
}

// pass 2: s_part[g * N + t] = sum over the group's rows of exp(x - M) / L, t < N, for the
// blocks [wgi * bpw, ..) of the coded keys of head g; (M, L) per row from the nw1 pass-1
// partials.  Grid (nw, G).
template <bool F32>
__global__ __launch_bounds__(SL_THREADS, 4) void sal_colsum(const void* __restrict__ K,
                                                            const void* __restrict__ Qw,
                                                            int64_t n, int G, int H, int w,
                                                            const float2* __restrict__ stats, int nw1,
                                                            float* __restrict__ s_part, int bpw) {
    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
    constexpr int KB = sl_keys<F32>();
    constexpr int TPB = KB / 16;
    __shared__ float colsum[SL_WAVES][KB];
    __shared__ float2 rowml[SL_WAVES * SL_MAX_RT * 16];   // (M, 1/L) of the head's rows
    const int wgi = blockIdx.x, g = blockIdx.y;
    const int64_t N = n - w;
    const int hpg = H / G, rows = hpg * w, nrt = (rows + 15) / 16;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int lane = threadIdx.x & 63;
    const int nblk = (int)((N + KB - 1) / KB);
    const int b0 = wgi * bpw, b1 = b0 + bpw < nblk ? b0 + bpw : nblk;

    u32x4 qh[SL_MAX_RT][4], ql[SL_MAX_RT][4];
    float rm[SL_MAX_RT][4], rinv[SL_MAX_RT][4];
#pragma unroll
    for (int j = 0; j < SL_MAX_RT; ++j) {
        const int rt = wave + SL_WAVES * j;
        if (rt < nrt) sl_qfrag<F32>(Qw, H, w, hpg, g, rows, rt, qh[j], ql[j]);
    }
    // Row statistics of head g from the pass-1 partials (every workgroup of the head forms
    // them): tpr threads per row, each over every tpr-th partial.  The partial loads issue
    // together, before the first two key blocks are requested, so the two round trips overlap.
    int tpr = 2;
    while (tpr * 2 * rows <= SL_THREADS && tpr < 64) tpr *= 2;
    const int r = threadIdx.x / tpr, h = threadIdx.x % tpr;
    const bool live = r < rows;
    const float2* st = stats + ((int64_t)g * rows + (live ? r : 0)) * nw1;
    float2 part[SL_MERGE_REG];
#pragma unroll
    for (int i = 0; i < SL_MERGE_REG; ++i) {
        const int b = h + tpr * i;
        part[i] = st[b < nw1 ? b : 0];
        if (!(b < nw1)) part[i].x = -INFINITY;
    }
    // The block loads are issued in asm after every compiler-visible load, so the compiler's
    // waits for the partials (counted over its own loads only) can only over-wait.
    sl_prime<F32>(lds, K, n, G, g, b0, b1);
    {
        // partials past the first SL_MERGE_REG of this thread (many rows x many pass-1
        // workgroups) come in batches of SL_MERGE_REG loads issued together, in the same
        // order as the first batch, so the sums keep one fixed order
        float mm = -INFINITY;
#pragma unroll
        for (int i = 0; i < SL_MERGE_REG; ++i) mm = fmaxf(mm, part[i].x);
        for (int b0 = h + tpr * SL_MERGE_REG; b0 < nw1; b0 += tpr * SL_MERGE_REG) {
            float x[SL_MERGE_REG];
#pragma unroll
            for (int i = 0; i < SL_MERGE_REG; ++i) {
                const int b = b0 + tpr * i;
                x[i] = st[b < nw1 ? b : 0].x;
            }
#pragma unroll
            for (int i = 0; i < SL_MERGE_REG; ++i)
                if (b0 + tpr * i < nw1) mm = fmaxf(mm, x[i]);
        }
        for (int off = 1; off < tpr; off <<= 1) mm = fmaxf(mm, shfl_xor_f(mm, off));
        float ll = 0.f;
        if (mm != -INFINITY) {
#pragma unroll
            for (int i = 0; i < SL_MERGE_REG; ++i)
                ll += part[i].x == -INFINITY ? 0.f : part[i].y * fast_exp(part[i].x - mm);
            for (int b0 = h + tpr * SL_MERGE_REG; b0 < nw1; b0 += tpr * SL_MERGE_REG) {
                float2 v[SL_MERGE_REG];
#pragma unroll
                for (int i = 0; i < SL_MERGE_REG; ++i) {
                    const int b = b0 + tpr * i;
                    v[i] = st[b < nw1 ? b : 0];
                }
#pragma unroll
                for (int i = 0; i < SL_MERGE_REG; ++i)
                    if (b0 + tpr * i < nw1) ll += v[i].x == -INFINITY ? 0.f : v[i].y * fast_exp(v[i].x - mm);
            }
        }
        for (int off = 1; off < tpr; off <<= 1) ll += shfl_xor_f(ll, off);
        if (live && h == 0) rowml[r] = make_float2(mm, 1.f / ll);
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < SL_MAX_RT; ++j) {
        const int rt = wave + SL_WAVES * j;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int rho = rt * 16 + (lane >> 4) * 4 + v;
            const bool ok = rt < nrt && rho < rows;
            const float2 mlv = rowml[ok ? rho : 0];
            rm[j][v] = mlv.x * 1.4426950408889634f;          // log2 units
            rinv[j][v] = ok ? mlv.y : 0.f;                   // rows past `rows` weigh nothing
        }
    }
    const float sl2 = 0.08838834764831845f * 1.4426950408889634f;   // log2(e) / sqrt(128)

    sl_pipeline<F32>(lds, K, n, G, g, b0, b1, [&](int b, const uint8_t* buf) {
        const int64_t k0 = (int64_t)b * KB;
        const int64_t kend = k0 + KB < N ? k0 + KB : N;
        const int ntile = (int)((kend - k0 + 15) / 16);
#pragma unroll
        for (int kt = 0; kt < TPB; ++kt) {
            if (kt >= ntile) break;
            float acc = 0.f;   // this lane's key column: sum over the wave's rows
#pragma unroll
            for (int j = 0; j < SL_MAX_RT; ++j) {
                const int rt = wave + SL_WAVES * j;
                if (rt >= nrt) continue;
                const f32x4 c = sl_logits<F32>(buf, kt, qh[j], ql[j]);
#pragma unroll
                for (int v = 0; v < 4; ++v) acc += __builtin_amdgcn_exp2f(c[v] * sl2 - rm[j][v]) * rinv[j][v];
            }
            acc = xsum32(xsum16(acc));
            if (lane < 16) colsum[wave][kt * 16 + lane] = acc;
        }
        __syncthreads();
        for (int kk = threadIdx.x; kk < ntile * 16; kk += SL_THREADS) {
            const int64_t t = k0 + kk;
            if (t < kend) {
                float s = 0.f;
#pragma unroll
                for (int ww = 0; ww < SL_WAVES; ++ww) s += colsum[ww][kk];
                s_part[(int64_t)g * N + t] = s;
            }
        }
    });
}

// pool: sbar[t] = (s_{t-2} + ... + s_{t+2}) / 5 with s_k = sum_g s_part[g][k] / (w H).  A
// block of 256 tokens first forms s for its tokens and a 2-token halo on each side.
constexpr int SP_T = 256;
__global__ __launch_bounds__(SP_T) void sal_pool(const float* __restrict__ s_part, int64_t N, int G,
                                                 float inv_wh, float* __restrict__ sbar) {
    __shared__ double sv[SP_T + 4];
    const int64_t t0 = (int64_t)blockIdx.x * SP_T;
    for (int i = threadIdx.x; i < SP_T + 4; i += SP_T) sv[i] = pool_term(s_part, N, G, inv_wh, t0 - 2 + i);
    __syncthreads();
    const int64_t t = t0 + threadIdx.x;
    if (t >= N) return;
    sbar[t] = pool5(sv, threadIdx.x + 2);
}

// ----------------------------------------------------------------------------------------
// Work split: a pass over nblk blocks of each of the G heads uses about SL_SLOTS workgroups,
// each taking bpw consecutive blocks of one head.
struct SalPlan {
    int nw, bpw;
};
static SalPlan sal_plan(int64_t nblk, int G) {
    int per_head = SL_SLOTS / G;
    per_head = per_head < 1 ? 1 : per_head;
    SalPlan p;
    p.bpw = (int)((nblk + per_head - 1) / per_head);
    p.bpw = p.bpw < 1 ? 1 : p.bpw;
    p.nw = (int)((nblk + p.bpw - 1) / p.bpw);
    return p;
}
static int sal_kb(const varrate_shape& sh) { return sh.dtype == VARRATE_BF16 ? sl_keys<false>() : sl_keys<true>(); }

size_t salience_ws_bytes(const varrate_shape& sh) {
    const int rows = (sh.H / sh.G) * sh.w;
    const int KB = sal_kb(sh);
    const SalPlan p1 = sal_plan((sh.n + KB - 1) / KB, sh.G);
    const int64_t N = sh.n - sh.w;
    return align256((size_t)sh.G * rows * p1.nw * sizeof(float2)) +
           align256((size_t)sh.G * N * sizeof(float));
}

template <bool F32>
static hipError_t sal_attr() {
    hipError_t e = ensure_lds_limit((const void*)sal_rowstats<F32>, 2 * SL_STAGE);
    if (e == hipSuccess) e = ensure_lds_limit((const void*)sal_colsum<F32>, 2 * SL_STAGE);
    return e;
}

const float* salience_part(const varrate_shape& sh, const uint8_t* ws) {
    const int rows = (sh.H / sh.G) * sh.w;
    const SalPlan p1 = sal_plan((sh.n + sal_kb(sh) - 1) / sal_kb(sh), sh.G);
    return (const float*)(ws + align256((size_t)sh.G * rows * p1.nw * sizeof(float2)));
}

float salience_pool_scale(const varrate_shape& sh) { return 1.0f / ((float)sh.w * (float)sh.H); }

hipError_t launch_salience(const varrate_shape& sh, const void* K, const void* Qw, float* sbar,
                           uint8_t* ws, hipStream_t st, bool pool) {
    const int rows = (sh.H / sh.G) * sh.w;
    const int64_t N = sh.n - sh.w;
    const int KB = sal_kb(sh);
    const SalPlan p1 = sal_plan((sh.n + KB - 1) / KB, sh.G);
    const SalPlan p2 = sal_plan((N + KB - 1) / KB, sh.G);
    float2* stats = (float2*)ws;
    ws += align256((size_t)sh.G * rows * p1.nw * sizeof(float2));
    float* s_part = (float*)ws;
    const bool bf = sh.dtype == VARRATE_BF16;
    hipError_t e = bf ? sal_attr<false>() : sal_attr<true>();
    if (e != hipSuccess) return e;
    dim3 g1(p1.nw, sh.G), g2(p2.nw, sh.G);
    const size_t lds = 2 * SL_STAGE;
    if (bf) {
        sal_rowstats<false><<<g1, SL_THREADS, lds, st>>>(K, Qw, sh.n, sh.G, sh.H, sh.w, stats, p1.nw, p1.bpw);
        sal_colsum<false><<<g2, SL_THREADS, lds, st>>>(K, Qw, sh.n, sh.G, sh.H, sh.w, stats, p1.nw, s_part, p2.bpw);
    } else {
        sal_rowstats<true><<<g1, SL_THREADS, lds, st>>>(K, Qw, sh.n, sh.G, sh.H, sh.w, stats, p1.nw, p1.bpw);
        sal_colsum<true><<<g2, SL_THREADS, lds, st>>>(K, Qw, sh.n, sh.G, sh.H, sh.w, stats, p1.nw, s_part, p2.bpw);
    }
    if (pool)
        sal_pool<<<(unsigned)((N + SP_T - 1) / SP_T), SP_T, 0, st>>>(s_part, N, sh.G, salience_pool_scale(sh), sbar);
    return hipGetLastError();
}

}  // namespace vr
