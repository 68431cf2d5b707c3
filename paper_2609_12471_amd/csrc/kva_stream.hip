// Plain streaming read of a device buffer: the achievable HBM read bandwidth
// for the decode kernels' loads (16-byte non-temporal), measured beside them.
// Each block XOR-reduces its share of the buffer and writes one word, so no
// load can be dropped.

#include "kva_internal.h"
#include "kva_device.h"

namespace kva {
namespace {

using namespace dev;

constexpr int kStreamThreads = 256;
constexpr int kStreamUnroll = 4;       // 16-byte loads in flight per lane

// Each wave streams one contiguous share of the buffer, 1 KiB per load
// instruction (a grid-stride loop measured 6.3-6.9 TB/s on MI355X, contiguous
// shares over 2048 waves 7.06 TB/s).
__global__ __launch_bounds__(kStreamThreads) void stream_read_kernel(const u32x4_t *src, int64_t n16,
                                                                     int64_t per_wave16, uint32_t *sink) {
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * (kStreamThreads / 64) + (threadIdx.x >> 6);
    const int64_t b = w * per_wave16;
    const int64_t e = min(b + per_wave16, n16);
    uint32_t x = 0;
    int64_t i = b + lane;
    for (; i + (kStreamUnroll - 1) * 64 < e; i += kStreamUnroll * 64) {
        u32x4_t v[kStreamUnroll];
#pragma unroll
        for (int u = 0; u < kStreamUnroll; ++u) v[u] = __builtin_nontemporal_load(src + i + u * 64);
#pragma unroll
        for (int u = 0; u < kStreamUnroll; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < e; i += 64) {
        const u32x4_t v = __builtin_nontemporal_load(src + i);
        x ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    // block XOR: waves by lane shuffles, then the four wave results in LDS
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) x ^= (uint32_t)__shfl_xor((int)x, d, 64);
    __shared__ uint32_t s_w[kStreamThreads / 64];
    if (lane == 0) s_w[threadIdx.x >> 6] = x;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0;
#pragma unroll
        for (int k = 0; k < kStreamThreads / 64; ++k) t ^= s_w[k];
        sink[blockIdx.x] = t;
    }
}

// One wave per block: block b writes the XCD it runs on (the XCC_ID hardware
// register, bits 3:0) to out[b].
__global__ __launch_bounds__(64) void xcd_ids_kernel(int32_t *out, int nblocks) {
    if ((int)blockIdx.x >= nblocks) return;
    // s_getreg immediate: size - 1 in bits 15:11, offset in 10:6, register 20 (XCC_ID)
    const int id = (int)__builtin_amdgcn_s_getreg((3 << 11) | (0 << 6) | 20);
    if (threadIdx.x == 0) out[blockIdx.x] = id & 15;
}

}  // namespace

hipError_t launch_xcd_ids(int32_t *out, int nblocks, hipStream_t stream) {
    hipLaunchKernelGGL(xcd_ids_kernel, dim3((unsigned)nblocks), dim3(64), 0, stream, out, nblocks);
    return hipGetLastError();
}

hipError_t launch_stream_read(const void *src, int64_t bytes, uint32_t *sink, int blocks,
                              hipStream_t stream) {
    const int64_t n16 = bytes / 16;
    const int64_t waves = (int64_t)blocks * (kStreamThreads / 64);
    const int64_t per_wave16 = (n16 + waves - 1) / waves;
    hipLaunchKernelGGL(stream_read_kernel, dim3((unsigned)blocks), dim3(kStreamThreads), 0, stream,
                       static_cast<const u32x4_t *>(src), n16, per_wave16, sink);
    return hipGetLastError();
}

}  // namespace kva
