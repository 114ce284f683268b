// HBM streaming-read probe: the rate a plain read stream of the weight-stream access pattern reaches on
// this part (one contiguous 1 KiB block per wavefront load, several loads in flight per lane).  A
// measurement aid for the roofline fractions the benchmark reports; not a step of the method.
#include "../../include/nld.h"
#include "nld_internal.h"

#include <hip/hip_runtime.h>

namespace nld {

// Workgroup b reads blocks [b * per, min((b + 1) * per, n_blocks)) of 1 KiB, wavefront w taking blocks
// w, w + waves, ... of that range, DEPTH loads per lane issued before any is consumed.  The XOR of
// everything read goes to sink[b], so no load can be dropped.
template <int DEPTH>
__global__ void __launch_bounds__(1024) hbm_read_probe_kernel(const uint4* buf, size_t n_blocks, size_t per,
                                                              uint32_t* sink) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, waves = blockDim.x >> 6;
    const size_t b0 = (size_t)blockIdx.x * per;
    const size_t b1 = b0 + per < n_blocks ? b0 + per : n_blocks;
    uint32_t acc = 0u;
    size_t blk = b0 + wave;
    const size_t step = (size_t)waves;
    for (; blk + (DEPTH - 1) * step < b1; blk += DEPTH * step) {
        uint4 v[DEPTH];
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) v[d] = buf[(blk + d * step) * 64 + lane];
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) acc ^= v[d].x ^ v[d].y ^ v[d].z ^ v[d].w;
    }
    for (; blk < b1; blk += step) {
        const uint4 v = buf[blk * 64 + lane];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) acc ^= __shfl_xor(acc, off);
    __shared__ uint32_t red[16];
    if (lane == 0) red[wave] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t t = 0u;
        for (int w = 0; w < waves; ++w) t ^= red[w];
        sink[blockIdx.x] = t;
    }
}

}  // namespace nld

extern "C" nld_status nld_hbm_read_probe(const void* buf, size_t bytes, int32_t grid, int32_t waves, int32_t depth,
                                         uint32_t* sink, void* stream) {
    using namespace nld;
    if (!buf || !sink) return NLD_ERR_INVALID_ARG;
    if (bytes < 1024 || bytes % 1024 || grid < 1 || waves < 1 || waves > 16) return NLD_ERR_INVALID_ARG;
    const size_t n_blocks = bytes / 1024;
    const size_t per = (n_blocks + grid - 1) / grid;
    const dim3 g((unsigned)grid), b((unsigned)(64 * waves));
    hipStream_t s = (hipStream_t)stream;
    switch (depth) {
        case 4: hbm_read_probe_kernel<4><<<g, b, 0, s>>>((const uint4*)buf, n_blocks, per, sink); break;
        case 8: hbm_read_probe_kernel<8><<<g, b, 0, s>>>((const uint4*)buf, n_blocks, per, sink); break;
        case 16: hbm_read_probe_kernel<16><<<g, b, 0, s>>>((const uint4*)buf, n_blocks, per, sink); break;
        case 32: hbm_read_probe_kernel<32><<<g, b, 0, s>>>((const uint4*)buf, n_blocks, per, sink); break;
        default: return NLD_ERR_INVALID_ARG;
    }
    return hipGetLastError() == hipSuccess ? NLD_OK : NLD_ERR_HIP;
}
