// Measurement aid: a plain streaming read of a device buffer, the practical
// HBM read ceiling the pool scan is compared with.  Each workgroup reads one
// contiguous stretch of the buffer; per step its 256 lanes issue U 16-byte
// non-temporal loads each, U consecutive 4 KiB stripes of the stretch.  The
// words are folded with XOR and one 64-bit word per workgroup is XOR-ed into
// the sink, so the loads cannot be dropped.  Few long stretches read fastest:
// on 8 GiB, 512 workgroups x 8 loads in flight reach 7.24 TB/s, 256 x 16 the
// same, 1024 x 8 6.88, 2048 x 8 6.51, and a grid-stride loop over 8192
// workgroups 6.1 (each stretch keeps DRAM rows open longer).
#include "common.hpp"
#include "internal.hpp"

#ifndef OIL_RS_U
#define OIL_RS_U 8
#endif
#ifndef OIL_RS_BLOCKS
#define OIL_RS_BLOCKS 512
#endif

namespace oil {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void read_stream_kernel(const u32x4* __restrict__ buf, int64_t n16,
                                                          int64_t per_block, unsigned long long* __restrict__ sink)
{
    constexpr int kU = OIL_RS_U;
    const int64_t lo = (int64_t)blockIdx.x * per_block;
    const int64_t hi = lo + per_block < n16 ? lo + per_block : n16;
    u32x4 acc = {0u, 0u, 0u, 0u};
    int64_t i = lo + threadIdx.x;
    for (; i + (kU - 1) * 256 < hi; i += kU * 256) {
        u32x4 v[kU];
#pragma unroll
        for (int u = 0; u < kU; u++)
            v[u] = __builtin_nontemporal_load(buf + i + u * 256);
#pragma unroll
        for (int u = 0; u < kU; u++)
            acc ^= v[u];
    }
    for (; i < hi; i += 256)
        acc ^= __builtin_nontemporal_load(buf + i);
    // little-endian: .x, .z are the low halves of the two 64-bit words, .y, .w the high halves
    unsigned long long w = ((unsigned long long)(acc.y ^ acc.w) << 32) | (acc.x ^ acc.z);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
        w ^= __shfl_xor(w, o, kWave);
    __shared__ unsigned long long part[4];
    if ((threadIdx.x & 63) == 0)
        part[threadIdx.x >> 6] = w;
    __syncthreads();
    if (threadIdx.x == 0)
        atomicXor(sink, part[0] ^ part[1] ^ part[2] ^ part[3]);
}

hipError_t launch_read_stream(const void* buf, int64_t n16, uint64_t* sink, hipStream_t stream)
{
    if (n16 <= 0)
        return hipSuccess;
    // contiguous stretches of whole 256-word (4 KiB) stripes, at most OIL_RS_BLOCKS workgroups
    const int64_t stripes = (n16 + 255) / 256;
    const int64_t blocks = stripes < OIL_RS_BLOCKS ? stripes : OIL_RS_BLOCKS;
    const int64_t per_block = (stripes + blocks - 1) / blocks * 256;
    const int64_t grid = (n16 + per_block - 1) / per_block;
    hipLaunchKernelGGL(read_stream_kernel, dim3((unsigned)grid), dim3(256), 0, stream, (const u32x4*)buf, n16,
                       per_block, (unsigned long long*)sink);
    return hipGetLastError();
}

}  // namespace oil
