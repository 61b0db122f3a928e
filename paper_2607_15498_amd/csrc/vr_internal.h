// Internal declarations shared by the HIP sources of libvarrate.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "varrate.h"
#include "vr_device.h"

namespace vr {

constexpr int CHUNK = VARRATE_CHUNK;
constexpr int64_t MAX_CODED = 1 << 20;   // allocator limits: chunk table in LDS, 24-bit index keys
constexpr int MAX_CODED_CHUNKS = (int)(MAX_CODED / CHUNK);

inline size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

// Raises kernel `fn`'s dynamic-LDS limit to at least `bytes` on the current device.  The
// raised limit is remembered per (kernel, device) under a lock, so concurrent callers and
// several devices are safe; this is the only state the library keeps across calls.
hipError_t ensure_lds_limit(const void* fn, size_t bytes);

// Residual codec: anchors are the prefix tokens 0, delta, ...; the coded tokens the rest.
inline int64_t anchor_count(const varrate_shape& sh) {
    return sh.anchor_stride > 0 ? (sh.n - sh.w + sh.anchor_stride - 1) / sh.anchor_stride : 0;
}
inline int64_t coded_count(const varrate_shape& sh) { return sh.n - sh.w - anchor_count(sh); }
// Eq. (3) with n_ref = anchors + window
inline int64_t coded_budget(const varrate_shape& sh) {
    return varrate_coded_budget(sh.n, sh.d, sh.w, sh.kappa_pct) - anchor_count(sh) * sh.d;
}
// The shape the coded-token stages see (allocation, projection, decode): the coded tokens
// followed by the window.  Its budget comes from the cache (cache.B), not from its kappa.
inline varrate_shape coded_shape(const varrate_shape& sh) {
    varrate_shape c = sh;
    c.n = coded_count(sh) + sh.w;
    c.anchor_stride = 0;
    return c;
}
struct AnchorWs {
    float* sbar;          // [n - w] pooled salience of the whole prefix
    float* sbar_c;        // [N] coded tokens' salience
    float* nrm;           // [na]
    float* pk;            // [n_atiles][N][4]
    uint32_t* pa;         // [n_atiles][N][4]
    uint16_t* nn;         // [N][4]
    void* Kr;             // [N + w][G][d] residuals, then the window rows
    void* Vr;
    uint32_t* cnt;        // [na]
    uint8_t* sal;         // salience workspace
    uint8_t* alloc;       // allocation workspace
};
size_t anchor_ws_bytes(const varrate_shape& sh);
AnchorWs anchor_ws(const varrate_shape& sh, uint8_t* ws);
hipError_t launch_anchor_search(const varrate_shape& sh, const void* K, const void* V, uint16_t* nn,
                                const AnchorWs& w, hipStream_t st);
hipError_t launch_anchor_encode(const varrate_shape& sh, const void* K, const void* V, const float* sbar,
                                const uint16_t* nn, const float* PK, const float* PV, varrate_cache& c,
                                const AnchorWs& w, hipStream_t st);

// Rotary keys: theta / (2 pi) per pair as a double-float (hi + lo), for the kernel arguments
struct RopeFreq { float hi[D / 2], lo[D / 2]; };
RopeFreq rope_freq(const varrate_shape& sh);
// Kr [n][G][d] = K with rows t < N turned back by -t (rounded to dtype), rows >= N copied
hipError_t launch_rope_unrotate(const varrate_shape& sh, const void* K, void* Kr, hipStream_t st);
// decode operands: basis fragments [G][4][8][2][64] u32x4 and the frequency table [128] fp32
constexpr size_t ROPE_FRAG_BYTES = (size_t)4 * 8 * 2 * 64 * 16;   // per KV head
hipError_t launch_rope_prep(const varrate_shape& sh, const float* PK, void* frags, float* freq, hipStream_t st);

// shared cross-head basis
hipError_t launch_allocate_joint(const varrate_shape& sh, int R, int64_t B, const float* sbar, uint16_t* rank,
                                 uint32_t* offset, uint32_t* chunk_off, uint8_t* ws, hipStream_t st,
                                 const float* s_part);
hipError_t launch_joint_project(const varrate_shape& sh, int R, const void* K, const void* V, const float* W,
                                const uint16_t* rank, const uint32_t* offset, void* coef, hipStream_t st);
size_t joint_decode_ws_bytes(const varrate_shape& sh, int R, int S, int Q);
hipError_t launch_joint_window(const varrate_shape& sh, const void* K, const void* V, varrate_jcache& c,
                               hipStream_t st);
hipError_t launch_joint_decode(const varrate_shape& sh, int R, const varrate_jcache* caches, int S, const void* q,
                               int Q, const float* W, void* out, uint8_t* ws, hipStream_t st);

size_t salience_ws_bytes(const varrate_shape& sh);
size_t allocate_ws_bytes(const varrate_shape& sh);
size_t decode_ws_bytes(const varrate_shape& sh, int S, int Q);
size_t decode_units(const varrate_shape& sh, int S, int Q);   // sequences x KV heads x row tiles
bool decode_supported(const varrate_shape& sh, int S, int Q);

// pool = false leaves the per-head column sums in the workspace (salience_part) for
// launch_allocate to pool (compress path: one launch fewer)
hipError_t launch_salience(const varrate_shape& sh, const void* K, const void* Qw, float* sbar,
                           uint8_t* ws, hipStream_t st, bool pool = true);
const float* salience_part(const varrate_shape& sh, const uint8_t* ws);
float salience_pool_scale(const varrate_shape& sh);
// s_part non-NULL: the first pass pools sbar from the column sums (and writes it) itself.
// chunk_sizes NULL: the chunk table c.chunk_off is scanned before return (the allocation entry
// point); non-NULL: it receives the workspace array of unscanned chunk sizes and c.chunk_off is
// left to the projection, which must then be given that array (compress path: one launch fewer)
hipError_t launch_allocate(const varrate_shape& sh, const float* sbar, varrate_cache& c,
                           uint8_t* ws, hipStream_t st, const float* s_part = nullptr,
                           const uint32_t** chunk_sizes = nullptr);
// chunk_sizes non-NULL: the chunk offsets are scanned from these sizes and written to
// c.chunk_off by the projection itself
hipError_t launch_project(const varrate_shape& sh, const void* K, const void* V, const float* PK,
                          const float* PV, varrate_cache& c, hipStream_t st,
                          const uint32_t* chunk_sizes = nullptr);
// reuse_group_region: every launch group (DC_SEQ sequences) writes its partial records to the
// start of `ws` instead of a region of its own (the no-allocation entry point)
// qcaches non-NULL: the coefficients are the quantised codes of qcaches[s] (same bits)
hipError_t launch_decode(const varrate_shape& sh, const varrate_cache* caches, int S, const void* q,
                         int Q, const float* PK, const float* PV, void* out, uint8_t* ws,
                         hipStream_t st, bool reuse_group_region = false,
                         const varrate_qcache* qcaches = nullptr);
size_t qcache_stride(const varrate_shape& sh, int bits);
hipError_t launch_quantize(const varrate_shape& sh, const varrate_cache& c, varrate_qcache& q, hipStream_t st);
// bytes of partial records one launch group needs (what the fixed scratch must hold)
size_t decode_group_bytes(const varrate_shape& sh, int S, int Q);
// this device's address of the fixed decode scratch array (looked up once per device)
hipError_t decode_scratch(uint8_t** out);
// streaming-read probe (measurement aid)
hipError_t launch_read_probe(const void* src, size_t bytes, uint32_t* sink, hipStream_t st);

}  // namespace vr
