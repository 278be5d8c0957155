// Attention-window stand-in, calibration copy and read-stream kernels, and event/stream
// helpers.
#include <hip/hip_runtime.h>

#include <cmath>

#include "common.h"
#include "ffn_device.h"

namespace {

using apex::ffn::ld_stream;

// Spins one wavefront until `ticks` of the constant-rate device clock have passed.
// The iteration cap only guards against a clock that fails to advance.
__global__ void spin_kernel(uint64_t ticks) {
    const uint64_t t0 = wall_clock64();
    for (uint64_t it = 0; it < (ticks + 1) * 4096ull; ++it)
        if (wall_clock64() - t0 >= ticks) break;
}

__global__ __launch_bounds__(256) void copy_kernel(uint4 *__restrict__ dst,
                                                   const uint4 *__restrict__ src, size_t n) {
    const size_t stride = size_t(gridDim.x) * blockDim.x;
    for (size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride)
        dst[i] = src[i];
}

// Reads n 16-byte chunks with four loads in flight per thread and folds them into one
// word per workgroup (so the loads cannot be dropped); the fold is the only write.  The
// loads are non-temporal, as the expert FFN's weight loads are.
__global__ __launch_bounds__(256) void read_kernel(const uint4 *__restrict__ src, size_t n,
                                                   uint32_t *__restrict__ sink) {
    const size_t stride = size_t(gridDim.x) * blockDim.x;
    uint32_t acc = 0;
    size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
    for (; i + 3 * stride < n; i += 4 * stride) {
        const uint4 a = ld_stream(src + i), b = ld_stream(src + i + stride),
                    c = ld_stream(src + i + 2 * stride), d = ld_stream(src + i + 3 * stride);
        acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^
               d.z ^ d.w;
    }
    for (; i < n; i += stride) {
        const uint4 a = ld_stream(src + i);
        acc ^= a.x ^ a.y ^ a.z ^ a.w;
    }
    for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o, 64);
    __shared__ uint32_t part[4];
    if (threadIdx.x % 64 == 0) part[threadIdx.x / 64] = acc;
    __syncthreads();
    if (threadIdx.x == 0) sink[blockIdx.x] = part[0] ^ part[1] ^ part[2] ^ part[3];
}

}  // namespace

extern "C" apex_status apex_spin_us(double us, hipStream_t stream) {
    APEX_REQUIRE(us >= 0.0 && us <= 1e6, "apex_spin_us: us=%g out of [0, 1e6]", us);
    if (us == 0.0) return APEX_OK;
    int dev = 0, khz = 0;
    APEX_HIP(hipGetDevice(&dev));
    APEX_HIP(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev));
    APEX_REQUIRE(khz > 0, "apex_spin_us: device reports no wall-clock rate");
    const uint64_t ticks = static_cast<uint64_t>(std::ceil(us * 1e-3 * double(khz)));
    hipLaunchKernelGGL(spin_kernel, dim3(1), dim3(64), 0, stream, ticks);
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}

extern "C" apex_status apex_copy_kernel(void *dst, const void *src, size_t bytes,
                                        hipStream_t stream) {
    APEX_REQUIRE(bytes % 16 == 0, "apex_copy_kernel: bytes=%zu not a multiple of 16", bytes);
    if (bytes == 0) return APEX_OK;
    APEX_REQUIRE(dst && src && apex::aligned16(dst) && apex::aligned16(src),
                 "apex_copy_kernel: NULL or misaligned pointer");
    const size_t n = bytes / 16;
    size_t blocks = (n + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(copy_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream,
                       static_cast<uint4 *>(dst), static_cast<const uint4 *>(src), n);
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}

extern "C" size_t apex_read_kernel_sink_words(size_t bytes) {
    const size_t n = bytes / 16;
    size_t blocks = (n + 1023) / 1024;
    return blocks < 1 ? 1 : (blocks > 1024 ? 1024 : blocks);
}

extern "C" apex_status apex_read_kernel(const void *src, size_t bytes, uint32_t *sink,
                                        hipStream_t stream) {
    APEX_REQUIRE(bytes % 16 == 0, "apex_read_kernel: bytes=%zu not a multiple of 16", bytes);
    if (bytes == 0) return APEX_OK;
    APEX_REQUIRE(src && sink && apex::aligned16(src), "apex_read_kernel: NULL or misaligned pointer");
    const size_t blocks = apex_read_kernel_sink_words(bytes);
    hipLaunchKernelGGL(read_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream,
                       static_cast<const uint4 *>(src), bytes / 16, sink);
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}

extern "C" apex_status apex_event_create(hipEvent_t *event, int timing) {
    APEX_REQUIRE(event, "apex_event_create: NULL out pointer");
    APEX_HIP(hipEventCreateWithFlags(event, timing ? hipEventDefault : hipEventDisableTiming));
    return APEX_OK;
}

extern "C" apex_status apex_event_destroy(hipEvent_t event) {
    APEX_REQUIRE(event, "apex_event_destroy: NULL event");
    APEX_HIP(hipEventDestroy(event));
    return APEX_OK;
}

extern "C" apex_status apex_event_record(hipEvent_t event, hipStream_t stream) {
    APEX_REQUIRE(event, "apex_event_record: NULL event");
    APEX_HIP(hipEventRecord(event, stream));
    return APEX_OK;
}

extern "C" apex_status apex_event_synchronize(hipEvent_t event) {
    APEX_REQUIRE(event, "apex_event_synchronize: NULL event");
    APEX_HIP(hipEventSynchronize(event));
    return APEX_OK;
}

extern "C" apex_status apex_event_elapsed_ms(hipEvent_t start, hipEvent_t stop, float *ms) {
    APEX_REQUIRE(start && stop && ms, "apex_event_elapsed_ms: NULL argument");
    APEX_HIP(hipEventElapsedTime(ms, start, stop));
    return APEX_OK;
}

extern "C" apex_status apex_stream_wait_event(hipStream_t stream, hipEvent_t event) {
    APEX_REQUIRE(event, "apex_stream_wait_event: NULL event");
    APEX_HIP(hipStreamWaitEvent(stream, event, 0));
    return APEX_OK;
}

extern "C" apex_status apex_stream_synchronize(hipStream_t stream) {
    APEX_HIP(hipStreamSynchronize(stream));
    return APEX_OK;
}
