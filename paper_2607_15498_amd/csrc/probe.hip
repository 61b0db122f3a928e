// Streaming-read probe: the read rate a plain kernel reaches on this device, measured beside
// the codec so the decode's fraction of the HBM peak can be set against what reading the
// same number of bytes takes.  Each workgroup reads one contiguous slice with eight 16-byte
// loads per lane in flight and folds the words into one value; the value is written only if
// it equals a fixed constant, which keeps the loads without writing anything in practice.
#include "vr_internal.h"

namespace vr {

constexpr int RP_T = 256;
constexpr int RP_U = 8;

__global__ __launch_bounds__(RP_T) void read_probe_kernel(const u32x4* __restrict__ src, size_t n16, size_t per16,
                                                          uint32_t* __restrict__ sink) {
    const size_t b0 = (size_t)blockIdx.x * per16;
    const size_t b1 = b0 + per16 < n16 ? b0 + per16 : n16;
    uint32_t acc = 0;
    for (size_t i = b0 + threadIdx.x; i < b1; i += (size_t)RP_T * RP_U) {
        u32x4 v[RP_U];
#pragma unroll
        for (int u = 0; u < RP_U; ++u) {
            const size_t j = i + (size_t)u * RP_T;
            v[u] = j < b1 ? src[j] : u32x4{0, 0, 0, 0};
        }
#pragma unroll
        for (int u = 0; u < RP_U; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
    }
    if (acc == 0x9E3779B9u) sink[blockIdx.x] = acc;
}

hipError_t launch_read_probe(const void* src, size_t bytes, uint32_t* sink, hipStream_t st) {
    const size_t n16 = bytes / 16;
    const size_t per16 = (n16 + VARRATE_PROBE_WGS - 1) / VARRATE_PROBE_WGS;
    read_probe_kernel<<<VARRATE_PROBE_WGS, RP_T, 0, st>>>(reinterpret_cast<const u32x4*>(src), n16, per16, sink);
    return hipGetLastError();
}

}  // namespace vr
