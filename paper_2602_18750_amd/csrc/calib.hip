// Roofline calibration, built as its own small library (libhill_calib.so) for
// the benchmark; not part of libhill or its ABI.  A plain streaming read of a
// device buffer, the fastest way this code base knows to pull a given number
// of bytes from HBM in one launch.  It computes nothing of the method; the
// benchmark times it at the scan's per-launch sizes to show what a single
// launch of that size can reach on this chip (launch, ramp and drain
// included).
#include <hip/hip_runtime.h>

#include "hill_device.h"

namespace {

constexpr int kCalibUnroll = 8;   // 16-byte loads in flight per thread

// Workgroup b reads the b-th contiguous share of the buffer, 256 lanes x 16 B
// per load round, kCalibUnroll rounds in flight.  The XOR of the words is
// stored only if it equals a constant, which keeps every load live without a
// store per workgroup.
__global__ __launch_bounds__(256) void calib_read_kernel(const uint4* __restrict__ p, int64_t n16,
                                                         uint32_t* __restrict__ sink)
{
    const int64_t per = (n16 + gridDim.x - 1) / gridDim.x;
    const int64_t b0 = static_cast<int64_t>(blockIdx.x) * per;
    const int64_t b1 = b0 + per < n16 ? b0 + per : n16;
    uint32_t acc = 0;
    for (int64_t i = b0 + threadIdx.x; i < b1; i += 256 * kCalibUnroll) {
        uint4 v[kCalibUnroll];
#pragma unroll
        for (int u = 0; u < kCalibUnroll; ++u) {
            const int64_t k = i + static_cast<int64_t>(u) * 256;
            v[u] = k < b1 ? hill::load_stream16(p + k) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < kCalibUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    if (acc == 0x9E3779B9u) sink[blockIdx.x] = acc;
}

}  // namespace

// One launch of `grid` workgroups reading the `bytes` bytes of the device
// buffer `buf` once.  buf 16-byte aligned, bytes a positive multiple of 16,
// 1 <= grid <= 65536, sink a device array of `grid` 32-bit words (its
// contents are meaningless).  Returns 0, 1 for an invalid argument (nothing
// launched), or 2 if the launch failed.
extern "C" __attribute__((visibility("default"))) int hill_calib_read(const void* buf, int64_t bytes, int32_t grid,
                                                                      uint32_t* sink, void* stream)
{
    if (!buf || !sink || (reinterpret_cast<uintptr_t>(buf) & 15u) || bytes < 16 || bytes % 16 || grid < 1 ||
        grid > 65536)
        return 1;
    hipLaunchKernelGGL(calib_read_kernel, dim3(grid), dim3(256), 0, static_cast<hipStream_t>(stream),
                       static_cast<const uint4*>(buf), bytes / 16, sink);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}
