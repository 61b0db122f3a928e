// Budgeted rank allocation (Sec. 3.2 Eq. (5), Algorithm 1 water-filling, integer ranks),
// exact integer arithmetic in a single workgroup, plus the chunk-local storage order.
//
// Weights.  u_t = 1 + floor(2^24 (sbar_t - min) / (max - min)) with each fp64 operation
// rounded once (all equal when max == min), so the ranks are a function of the fp32 input.
//
// Water level.  With D = R - r_min, E = B - N r_min, the excess handed out at level
// lambda = D / tau is F(tau) = D (tau c_ge(tau) + s_lt(tau)) / tau, where c_ge counts
// u >= tau and s_lt sums u < tau.  F falls as tau grows, so the integer
//     tau_lo = max{ tau in [1, u_max] : D (tau c_ge(tau) + s_lt(tau)) >= E tau }
// is found from two histogram levels of u (12 + 12 bits) evaluated at bin edges.  The
// tokens capped at R are exactly {u > tau_lo} (ties exactly at R stay uncapped), k of them;
// the others get q_t = r_min + u_t M / Q with M = B - R k - r_min (N - k), Q = sum of their u.
// This is the fixed point of Algorithm 1's clip-and-redistribute loop.
//
// Integer ranks.  floor(q_t) plus one unit for the rho = B - sum floor(q_t) uncapped tokens
// with the largest keys (phi_t = (u_t M) mod Q, then u_t, then lower index), found by a
// most-significant-digit radix select (11-bit digits, common-prefix skipping) over the
// 2 x 64-bit key.  All arithmetic is integer: the ranks are bit-exact and deterministic.
//
// Every pass over the N tokens keeps eight independent loads in flight per thread.  The
// selection's first digit comes from phi < Q directly; when the chosen bucket holds at most
// 2048 candidates they are gathered into LDS and the remaining digits never touch memory.
#include "vr_internal.h"

namespace vr {

constexpr int AL_T = 1024;
constexpr int AL_W = AL_T / 64;
constexpr int CBITS = 12;
constexpr int NBIN = (1 << CBITS) + 1;     // coarse bins of u (u <= 2^24 + 1)
constexpr uint64_t CAPPED = 1ull << 63;

template <typename T> __device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// Block exclusive scan of one value per thread; `tot` receives the block total.
template <typename T>
__device__ T block_exscan(T v, T* wtot, T& tot) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    T x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        T y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    if (lane == 63) wtot[wid] = x;
    __syncthreads();
    T pre = 0, all = 0;
    for (int i = 0; i < AL_W; ++i) {
        T wv = wtot[i];
        if (i < wid) pre += wv;
        all += wv;
    }
    __syncthreads();
    tot = all;
    return pre + x - v;
}

template <typename T, typename Op>
__device__ T block_reduce(T v, T* scratch, Op op) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = op(v, __shfl_xor(v, off, 64));
    if ((threadIdx.x & 63) == 0) scratch[threadIdx.x >> 6] = v;
    __syncthreads();
    T r = scratch[0];
    for (int i = 1; i < AL_W; ++i) r = op(r, scratch[i]);
    __syncthreads();
    return r;
}

// In-place exclusive scan of n (<= 4 * AL_T + 4) entries held in LDS; returns the total.
template <typename T>
__device__ T lds_exscan(T* a, int n, T* wtot) {
    const int per = (n + AL_T - 1) / AL_T;
    const int b = threadIdx.x * per;
    T loc = 0;
    for (int i = 0; i < per; ++i)
        if (b + i < n) loc += a[b + i];
    T tot;
    T pre = block_exscan<T>(loc, wtot, tot);
    for (int i = 0; i < per; ++i)
        if (b + i < n) {
            T v = a[b + i];
            a[b + i] = pre;
            pre += v;
        }
    __syncthreads();
    return tot;
}

struct SelState {
    uint64_t pv, pm;   // fixed prefix value / mask of the field being narrowed
    uint64_t T_hi, T_lo;
    int64_t need;
    int phase;         // 0: narrowing phi, 1: narrowing (u, ~t)
    int done;
    int ncand;         // candidates gathered into LDS
};

__device__ __forceinline__ uint64_t lo_key(uint32_t u, int64_t t) {
    return ((uint64_t)u << 24) | (uint64_t)(0xFFFFFFu - (uint32_t)t);
}

// Visit tokens t = tid, tid + AL_T, ... with U independent loads in flight per thread.
template <int U, class Load, class Proc>
__device__ __forceinline__ void sweep(int64_t N, Load load, Proc proc) {
    for (int64_t b = 0; b < N; b += (int64_t)U * AL_T) {
        decltype(load((int64_t)0)) v[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t t = b + (int64_t)k * AL_T + threadIdx.x;
            if (t < N) v[k] = load(t);
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t t = b + (int64_t)k * AL_T + threadIdx.x;
            if (t < N) proc(t, v[k]);
        }
    }
}

struct PhiU {
    uint64_t phi;
    uint32_t u;
};

struct Fin {
    uint64_t phi;
    uint32_t u;
    uint32_t r;
};

// Most-significant-digit radix narrowing of the selection threshold over the candidates
// enumerated by visit(f) (f(hi, lo) per uncapped candidate), starting from `sel`.
template <class Visit>
__device__ void radix_narrow(Visit visit, SelState& sel, uint32_t* cnt, uint32_t* wtot32,
                             unsigned long long* wtot64) {
    const int tid = threadIdx.x;
    while (!sel.done) {
        const int phase = sel.phase;
        const uint64_t pv = sel.pv, pm = sel.pm, T_hi = sel.T_hi;
        auto field = [&](uint64_t hi, uint64_t lo, uint64_t& f) -> bool {
            if (phase == 0) {
                f = hi;
            } else {
                if (hi != T_hi) return false;
                f = lo;
            }
            return (f & pm) == pv;
        };
        uint64_t fmn = ~0ull, fmx = 0;
        visit([&](uint64_t hi, uint64_t lo) {
            uint64_t f;
            if (field(hi, lo, f)) {
                fmn = f < fmn ? f : fmn;
                fmx = f > fmx ? f : fmx;
            }
        });
        fmn = block_reduce<unsigned long long>(fmn, wtot64, [](unsigned long long a, unsigned long long b) { return a < b ? a : b; });
        fmx = block_reduce<unsigned long long>(fmx, wtot64, [](unsigned long long a, unsigned long long b) { return a > b ? a : b; });
        if (fmn == fmx) {
            if (tid == 0) {
                if (phase == 0) {
                    sel.T_hi = fmn; sel.phase = 1; sel.pv = 0; sel.pm = 0;
                } else {
                    sel.T_lo = fmn; sel.done = 1;   // keys are unique: a single candidate
                }
            }
            __syncthreads();
            continue;
        }
        const int p = 63 - __clzll((long long)(fmn ^ fmx));
        const int sh = p > 10 ? p - 10 : 0;
        const uint64_t dmask = (1ull << (p - sh + 1)) - 1;
        const uint64_t above_mask = (p == 63) ? 0ull : ~((2ull << p) - 1);
        for (int i = tid; i < 2048; i += AL_T) cnt[i] = 0;
        __syncthreads();
        visit([&](uint64_t hi, uint64_t lo) {
            uint64_t f;
            if (field(hi, lo, f)) atomicAdd(&cnt[(f >> sh) & dmask], 1u);
        });
        __syncthreads();
        const int d0 = 2047 - 2 * tid, d1 = d0 - 1;
        const uint32_t c0 = cnt[d0], c1 = cnt[d1];
        uint32_t tot;
        const uint32_t above0 = block_exscan<uint32_t>(c0 + c1, wtot32, tot);
        const int64_t need = sel.need;
        __syncthreads();
        int hit = -1;
        uint32_t hit_above = 0, hit_cnt = 0;
        if ((int64_t)above0 < need && need <= (int64_t)(above0 + c0)) { hit = d0; hit_above = above0; hit_cnt = c0; }
        const uint32_t above1 = above0 + c0;
        if ((int64_t)above1 < need && need <= (int64_t)(above1 + c1)) { hit = d1; hit_above = above1; hit_cnt = c1; }
        if (hit >= 0) {
            const int64_t nn = need - (int64_t)hit_above;
            const uint64_t npv = (fmn & above_mask) | ((uint64_t)hit << sh);
            sel.need = nn;
            sel.pv = npv;
            sel.pm = ~((1ull << sh) - 1);
            if ((int64_t)hit_cnt == nn) {
                if (phase == 0) { sel.T_hi = npv; sel.T_lo = 0; }
                else { sel.T_lo = npv; }
                sel.done = 1;
            }
        }
        __syncthreads();
    }
}

constexpr int SEL_CAP = 2048;    // candidates the selection can finish in LDS

__global__ __launch_bounds__(AL_T) void alloc_kernel(const float* __restrict__ sbar, int64_t N,
                                                      int64_t B, int r_min, int R,
                                                      uint32_t* __restrict__ u_ws,
                                                      uint64_t* __restrict__ phi_ws,
                                                      uint8_t* __restrict__ rank,
                                                      uint32_t* __restrict__ chunk_off,
                                                      int n_chunks) {
    __shared__ uint32_t cnt[NBIN + 1];
    __shared__ unsigned long long sm[NBIN + 1];
    __shared__ unsigned long long wtot64[AL_W];
    __shared__ uint32_t wtot32[AL_W];
    __shared__ float redf[AL_W];
    __shared__ SelState sel;
    const int tid = threadIdx.x;
    constexpr int U = 8;

    // ---- 1. min / max of the pooled salience
    float mn = INFINITY, mx = -INFINITY;
    sweep<U>(N, [&](int64_t t) { return sbar[t]; }, [&](int64_t, float s) {
        mn = fminf(mn, s);
        mx = fmaxf(mx, s);
    });
    mn = block_reduce<float>(mn, redf, [](float a, float b) { return fminf(a, b); });
    mx = block_reduce<float>(mx, redf, [](float a, float b) { return fmaxf(a, b); });

    // ---- 2. integer weights + coarse histogram (count, sum) of u >> 12
    for (int i = tid; i <= NBIN; i += AL_T) { cnt[i] = 0; sm[i] = 0; }
    __syncthreads();
    const bool flat = !(mx > mn);
    const double lo = (double)mn;
    const double range = (double)mx - lo;
    uint32_t umax = 0;
    sweep<U>(N, [&](int64_t t) { return sbar[t]; }, [&](int64_t t, float s) {
        uint32_t u;
        if (flat) {
            u = (1u << 24) + 1u;
        } else {
            const double num = (double)s - lo;
            double shat = num / range;
            // non-finite inputs cannot index past the histograms
            shat = shat >= 0.0 ? (shat <= 1.0 ? shat : 1.0) : 0.0;
            u = 1u + (uint32_t)floor(shat * 16777216.0);
        }
        u_ws[t] = u;
        umax = u > umax ? u : umax;
        atomicAdd(&cnt[u >> CBITS], 1u);
        atomicAdd(&sm[u >> CBITS], (unsigned long long)u);
    });
    umax = block_reduce<uint32_t>(umax, wtot32, [](uint32_t a, uint32_t b) { return a > b ? a : b; });
    __syncthreads();

    const uint64_t Dr = (uint64_t)(R - r_min);
    const uint64_t E = (uint64_t)(B - N * (int64_t)r_min);
    const int nb = (int)(umax >> CBITS) + 1;
    // exclusive prefixes over bins 0..nb (entry nb = totals)
    lds_exscan<uint32_t>(cnt, nb + 1, wtot32);
    lds_exscan<unsigned long long>(sm, nb + 1, wtot64);
    // P'(tau) at coarse edges tau_b = max(1, b << 12): c_ge = N - cnt_ex[b], s_lt = sm_ex[b]
    int bbest = 0;
    for (int b = tid; b < nb; b += AL_T) {
        const uint64_t tau = b == 0 ? 1 : ((uint64_t)b << CBITS);
        const uint64_t cge = (uint64_t)N - cnt[b];
        const uint64_t slt = sm[b];
        if (Dr * (tau * cge + slt) >= E * tau) bbest = b > bbest ? b : bbest;
    }
    bbest = (int)block_reduce<uint32_t>((uint32_t)bbest, wtot32,
                                        [](uint32_t a, uint32_t b) { return a > b ? a : b; });
    const uint64_t cge_next = (uint64_t)N - cnt[bbest + 1];   // tokens in bins above bbest
    const uint64_t slt_b = sm[bbest];                          // sum of u in bins below bbest
    __syncthreads();

    // ---- 3. fine histogram of the low 12 bits inside bin bbest
    for (int i = tid; i <= NBIN; i += AL_T) { cnt[i] = 0; sm[i] = 0; }
    __syncthreads();
    sweep<U>(N, [&](int64_t t) { return u_ws[t]; }, [&](int64_t, uint32_t u) {
        if ((int)(u >> CBITS) == bbest) {
            atomicAdd(&cnt[u & ((1u << CBITS) - 1)], 1u);
            atomicAdd(&sm[u & ((1u << CBITS) - 1)], (unsigned long long)u);
        }
    });
    __syncthreads();
    const int nf = 1 << CBITS;
    lds_exscan<uint32_t>(cnt, nf + 1, wtot32);
    lds_exscan<unsigned long long>(sm, nf + 1, wtot64);
    const uint64_t fc_total = cnt[nf];
    const uint64_t base_tau = (uint64_t)bbest << CBITS;
    const int f_lo = bbest == 0 ? 1 : 0;
    const int f_hi = (int)(((uint64_t)umax - base_tau) < (uint64_t)(nf - 1) ? (umax - base_tau) : (nf - 1));
    int fbest = f_lo;
    for (int f = tid; f <= f_hi; f += AL_T) {
        if (f < f_lo) continue;
        const uint64_t tau = base_tau + f;
        const uint64_t cge = cge_next + fc_total - cnt[f];
        const uint64_t slt = slt_b + sm[f];
        if (Dr * (tau * cge + slt) >= E * tau) fbest = f > fbest ? f : fbest;
    }
    fbest = (int)block_reduce<uint32_t>((uint32_t)fbest, wtot32,
                                        [](uint32_t a, uint32_t b) { return a > b ? a : b; });
    const uint32_t tau_lo = (uint32_t)(base_tau + fbest);
    const int64_t kcap = (int64_t)(cge_next + fc_total - cnt[fbest + 1]);
    const uint64_t Q = slt_b + sm[fbest + 1];
    const int64_t M = B - (int64_t)R * kcap - (int64_t)r_min * (N - kcap);
    const double invQ = 1.0 / (double)Q;
    __syncthreads();

    // ---- 4. floors and fractional keys
    unsigned long long fsum = 0;
    sweep<U>(N, [&](int64_t t) { return u_ws[t]; }, [&](int64_t t, uint32_t u) {
        uint32_t base;
        uint64_t phi;
        if (u > tau_lo) {
            base = (uint32_t)R;
            phi = CAPPED;
        } else {
            // num < 2^52 and Q < 2^45 are exact in fp64; the reciprocal quotient is within
            // one unit of floor(num / Q) and the integer remainder corrects it exactly
            const uint64_t num = (uint64_t)u * (uint64_t)M;
            int64_t f = (int64_t)((double)num * invQ);
            int64_t rem = (int64_t)num - f * (int64_t)Q;
            if (rem < 0) { f -= 1; rem += (int64_t)Q; }
            if (rem >= (int64_t)Q) { f += 1; rem -= (int64_t)Q; }
            phi = (uint64_t)rem;
            base = (uint32_t)(r_min + f);
        }
        rank[t] = (uint8_t)base;
        phi_ws[t] = phi;
        fsum += base;
    });
    fsum = block_reduce<unsigned long long>(fsum, wtot64,
                                            [](unsigned long long a, unsigned long long b) { return a + b; });
    const int64_t rho = B - (int64_t)fsum;

    // ---- 5. select the rho largest (phi, u, -t) keys among uncapped tokens
    auto load_pu = [&](int64_t t) { return PhiU{phi_ws[t], u_ws[t]}; };
    if (tid == 0) {
        sel.pv = 0; sel.pm = 0; sel.T_hi = ~0ull; sel.T_lo = ~0ull;
        sel.need = rho; sel.phase = 0; sel.done = rho <= 0; sel.ncand = 0;
    }
    __syncthreads();
    if (!sel.done) {
        // first digit: phi < Q, so its top 11 significant bits need no range pass
        const uint64_t qm1 = Q > 1 ? Q - 1 : 1;
        const int qb = 64 - __clzll((long long)qm1);
        const int sh0 = qb > 11 ? qb - 11 : 0;
        for (int i = tid; i < 2048; i += AL_T) cnt[i] = 0;
        __syncthreads();
        sweep<U>(N, [&](int64_t t) { return phi_ws[t]; }, [&](int64_t, uint64_t phi) {
            if (phi != CAPPED) atomicAdd(&cnt[(phi >> sh0) & 2047], 1u);
        });
        __syncthreads();
        const int d0 = 2047 - 2 * tid, d1 = d0 - 1;
        const uint32_t c0 = cnt[d0], c1 = cnt[d1];
        uint32_t tot;
        const uint32_t above0 = block_exscan<uint32_t>(c0 + c1, wtot32, tot);
        const int64_t need = sel.need;
        __syncthreads();
        const uint32_t above1 = above0 + c0;
        int hit = -1;
        uint32_t hit_above = 0, hit_cnt = 0;
        if ((int64_t)above0 < need && need <= (int64_t)(above0 + c0)) { hit = d0; hit_above = above0; hit_cnt = c0; }
        if ((int64_t)above1 < need && need <= (int64_t)(above1 + c1)) { hit = d1; hit_above = above1; hit_cnt = c1; }
        if (hit >= 0) {
            const int64_t nn = need - (int64_t)hit_above;
            sel.need = nn;
            sel.pv = (uint64_t)hit << sh0;
            sel.pm = ~((1ull << sh0) - 1);
            if ((int64_t)hit_cnt == nn) { sel.T_hi = sel.pv; sel.T_lo = 0; sel.done = 1; }
            sel.ncand = (int)hit_cnt;
        }
        __syncthreads();
        if (!sel.done && sel.ncand <= SEL_CAP) {
            // gather the bucket's candidates into LDS and finish there
            unsigned long long* chi = sm;
            unsigned long long* clo = sm + SEL_CAP;
            const uint64_t pv = sel.pv, pm = sel.pm;
            __syncthreads();
            if (tid == 0) sel.ncand = 0;
            __syncthreads();
            sweep<U>(N, load_pu, [&](int64_t t, PhiU x) {
                if (x.phi != CAPPED && (x.phi & pm) == pv) {
                    const int slot = atomicAdd(&sel.ncand, 1);
                    chi[slot] = x.phi;
                    clo[slot] = lo_key(x.u, t);
                }
            });
            __syncthreads();
            const int nc = sel.ncand;
            radix_narrow([&](auto f) {
                for (int i = tid; i < nc; i += AL_T) f(chi[i], clo[i]);
            }, sel, cnt, wtot32, wtot64);
        } else if (!sel.done) {
            radix_narrow([&](auto f) {
                sweep<U>(N, load_pu, [&](int64_t t, PhiU x) {
                    if (x.phi != CAPPED) f(x.phi, lo_key(x.u, t));
                });
            }, sel, cnt, wtot32, wtot64);
        }
    }
    const uint64_t T_hi = sel.T_hi, T_lo = sel.T_lo;
    const bool any = rho > 0;

    // ---- 6. final ranks and chunk sums
    for (int i = tid; i < n_chunks; i += AL_T) cnt[i] = 0;
    __syncthreads();
    for (int64_t b = 0; b < N; b += (int64_t)U * AL_T) {
        Fin v[U];
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t t = b + (int64_t)k * AL_T + tid;
            if (t < N) v[k] = Fin{phi_ws[t], u_ws[t], rank[t]};
        }
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const int64_t t = b + (int64_t)k * AL_T + tid;
            uint32_t r = 0;
            if (t < N) {
                r = v[k].r;
                if (any && v[k].phi != CAPPED) {
                    const bool take = v[k].phi > T_hi || (v[k].phi == T_hi && lo_key(v[k].u, t) >= T_lo);
                    if (take) {
                        r += 1;
                        rank[t] = (uint8_t)r;
                    }
                }
            }
            // a wave covers 64 consecutive tokens, all inside one 256-token chunk
            const uint32_t ws = wave_sum(r);
            const int64_t tw = b + (int64_t)k * AL_T + (tid & ~63);
            if ((tid & 63) == 0 && tw < N) atomicAdd(&cnt[tw >> 8], ws);
        }
    }
    __syncthreads();
    const uint32_t total = lds_exscan<uint32_t>(cnt, n_chunks, wtot32);
    for (int i = tid; i < n_chunks; i += AL_T) chunk_off[i] = cnt[i];
    if (tid == 0) chunk_off[n_chunks] = total;
}

size_t allocate_ws_bytes(const varrate_shape& sh) {
    const int64_t N = sh.n - sh.w;
    return align256((size_t)N * sizeof(uint32_t)) + align256((size_t)N * sizeof(uint64_t));
}

hipError_t launch_allocate(const varrate_shape& sh, const float* sbar, varrate_cache& c,
                           uint8_t* ws, hipStream_t st) {
    const int64_t N = sh.n - sh.w;
    uint32_t* u_ws = (uint32_t*)ws;
    uint64_t* phi_ws = (uint64_t*)(ws + align256((size_t)N * sizeof(uint32_t)));
    const int n_chunks = (int)((N + CHUNK - 1) / CHUNK);
    alloc_kernel<<<1, AL_T, 0, st>>>(sbar, N, c.B, sh.r_min, D, u_ws, phi_ws, c.rank, c.chunk_off,
                                     n_chunks);
    return hipGetLastError();
}

}  // namespace vr
