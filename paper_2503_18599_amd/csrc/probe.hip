// Streaming-read probe: the HBM read bandwidth that plain loads reach on this device,
// measured beside the decode-attention kernel so that its achieved rate can be read
// against both the 8 TB/s peak and what simple loads attain.
//
// The pattern is n records of bytes_per_record bytes, record_stride bytes apart: one
// contiguous buffer (record_stride == bytes_per_record), or the first bytes of every page
// record of a cache pool, as decode attention reads them.  Every thread walks a flat list
// of 16-byte chunks (chunk i is chunk i mod c of record i / c, c chunks per record) with
// eight non-temporal loads in flight, so consecutive lanes read consecutive bytes; the
// record of a chunk comes from a multiply-high by a precomputed reciprocal.  All bytes are
// folded into an XOR checksum (one atomic per workgroup) so that no load can be dropped.
#include "oaken_internal.h"

namespace oaken {
namespace {

constexpr int kProbeUnroll = 8;
constexpr int kProbeBlocks = 2048;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void probe_read_kernel(ProbeArgs a) {
    const uint32_t total = a.total_chunks;
    const uint32_t nthr = gridDim.x * blockDim.x;
    uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    // record of chunk j: (j * magic) >> shift, exact for every j < 2^31
    auto addr = [&](uint32_t j) {
        const uint32_t r = (uint32_t)(((uint64_t)j * a.magic) >> a.shift);
        const uint32_t c = j - r * (uint32_t)a.chunks;
        return reinterpret_cast<const u32x4*>(a.base + (uint64_t)r * (uint64_t)a.record_stride + 16u * c);
    };
    uint32_t acc = 0;
    for (; i + (kProbeUnroll - 1) * nthr < total; i += kProbeUnroll * nthr) {
        u32x4 v[kProbeUnroll];
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) v[u] = __builtin_nontemporal_load(addr(i + u * nthr));
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
    }
    for (; i < total; i += nthr) {
        const u32x4 v = __builtin_nontemporal_load(addr(i));
        acc ^= v[0] ^ v[1] ^ v[2] ^ v[3];
    }
    __shared__ uint32_t part[4];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o, 64);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) atomicXor(a.checksum, part[0] ^ part[1] ^ part[2] ^ part[3]);
}

}  // namespace

bool prepare_probe(ProbeArgs& a) {
    const int64_t total = a.n_records * (int64_t)a.chunks;
    if (total <= 0 || total >= (int64_t(1) << 31)) return false;
    // multiply-high division by c for 31-bit dividends: l = ceil(log2 c),
    // magic = ceil(2^(31 + l) / c) < 2^32
    int l = 0;
    while ((int64_t(1) << l) < a.chunks) ++l;
    a.shift = 31 + l;
    a.magic = (uint32_t)(((uint64_t(1) << a.shift) + (uint64_t)a.chunks - 1) / (uint64_t)a.chunks);
    a.total_chunks = (uint32_t)total;
    return true;
}

hipError_t launch_probe_read(const ProbeArgs& a, hipStream_t st) {
    const uint32_t blocks = (uint32_t)std::min<int64_t>(kProbeBlocks, std::max<int64_t>(1, ((int64_t)a.total_chunks + 255) / 256));
    hipLaunchKernelGGL(probe_read_kernel, dim3(blocks), dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace oaken
