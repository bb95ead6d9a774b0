// On-demand sparse pages (the sparse management table of Sec. 5.2): the free list
// that the quantizer pops pages from, its reset, and the release of retired blocks.
//
// Free list (int32): [0] number of free pages n, [1] overflow flag, [2 .. 2+n) free
// page ids.  A record's table entry i is 1 + the id of the page holding bytes
// [256 i, 256 i + 256) of its COO stream, or 0 when the record holds no such page.
#include "oaken_internal.h"

#include <algorithm>

namespace oaken {
namespace {

// Every page free, overflow cleared, and every record of the dense pool emptied
// (counts and page table zeroed), so that no record claims a page.
__global__ __launch_bounds__(256) void sparse_reset_kernel(SparseArgs a) {
    const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t nthr = (int64_t)gridDim.x * blockDim.x;
    if (tid == 0) {
        a.sfree[0] = a.spages;
        a.sfree[1] = 0;
    }
    for (int64_t i = tid; i < a.spages; i += nthr) a.sfree[2 + i] = (int32_t)i;
    // per record: counts (cbytes) and the page table (tbytes), as dwords
    const int64_t nrec = (int64_t)a.num_blocks * a.H * 2;
    const int cw = a.cbytes / 4, tw = a.tbytes / 4;
    for (int64_t i = tid; i < nrec * (cw + tw); i += nthr) {
        const int64_t r = i / (cw + tw);
        const int w = (int)(i % (cw + tw));
        uint8_t* rec = a.pool + r * a.stride;
        int32_t* dst = w < cw ? reinterpret_cast<int32_t*>(rec) + w
                              : reinterpret_cast<int32_t*>(rec + a.table) + (w - cw);
        *dst = 0;
    }
}

// One wave per (block, KV head, K|V): push the record's pages back and empty it.
__global__ __launch_bounds__(64) void sparse_release_kernel(SparseArgs a, const int32_t* block_ids) {
    const int lane = threadIdx.x;
    const int blk = block_ids[blockIdx.x];
    if (blk < 0 || blk >= a.num_blocks) return;
    uint8_t* rec = a.pool + ((int64_t)blk * a.H * 2 + blockIdx.y) * a.stride;
    int32_t* tab = reinterpret_cast<int32_t*>(rec + a.table);
    const int nt = a.tbytes / 4;
    const int entry = lane < nt ? tab[lane] : 0;
    const bool held = entry > 0 && entry <= a.spages;
    const uint64_t hm = __ballot(held);
    const int k = __popcll(hm);
    int t = 0;
    if (k > 0 && lane == 0) t = atomicAdd(&a.sfree[0], k);
    t = __shfl(t, 0, 64);
    // (a consistent list has room for every held page; the bound only guards the array)
    const int r = __popcll(hm & ((1ull << lane) - 1ull));
    if (held && t + r < a.spages) a.sfree[2 + t + r] = entry - 1;
    if (lane < nt) tab[lane] = 0;
    if (lane < a.cbytes / 4) reinterpret_cast<int32_t*>(rec)[lane] = 0;
}

}  // namespace

hipError_t launch_sparse_reset(const SparseArgs& a, hipStream_t st) {
    const int64_t work = std::max<int64_t>(a.spages, (int64_t)a.num_blocks * a.H * 2 * ((a.cbytes + a.tbytes) / 4));
    const int blocks = (int)std::min<int64_t>(4096, std::max<int64_t>(1, (work + 255) / 256));
    hipLaunchKernelGGL(sparse_reset_kernel, dim3(blocks), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_sparse_release(const SparseArgs& a, const int32_t* block_ids, int n_blocks, hipStream_t st) {
    hipLaunchKernelGGL(sparse_release_kernel, dim3(n_blocks, a.H * 2), dim3(64), 0, st, a, block_ids);
    return hipGetLastError();
}

}  // namespace oaken
