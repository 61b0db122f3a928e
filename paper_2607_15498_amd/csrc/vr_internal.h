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
// s_part non-NULL: the first pass pools sbar from the column sums (and writes it) itself
hipError_t launch_allocate(const varrate_shape& sh, const float* sbar, varrate_cache& c,
                           uint8_t* ws, hipStream_t st, const float* s_part = nullptr);
hipError_t launch_project(const varrate_shape& sh, const void* K, const void* V, const float* PK,
                          const float* PV, varrate_cache& c, hipStream_t st);
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

}  // namespace vr
