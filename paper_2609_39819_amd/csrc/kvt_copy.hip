// Block-list copy between the HBM page pool and pinned host memory.
//
// The multi-tier cache moves whole pages between GPU HBM and host memory
// (offload of pages leaving HBM, reload of pages coming back).  One launch
// moves an arbitrary list of pages: the host side is a packed array
// [n][K | V][Hkv][16][D] in page-list order, the device side the pages
// block_ids[i] of the K and V pools.  The GPU reads and writes the pinned
// host buffer directly over the host link, so a scattered page list costs
// one launch instead of one DMA request per page.
//
// Work split: 16-byte pieces, consecutive threads take consecutive pieces of
// one page (a wave moves 1 KiB of contiguous bytes on both sides).
#include "kvt_internal.h"

namespace kvt {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void copy_blocks_kernel(const CopyArgs a) {
  const int64_t pieces = a.page_bytes / 16;               // per page per tensor
  const int64_t total = a.n * 2 * pieces;
  const uint32_t nb = (uint32_t)min<int64_t>(a.num_blocks, 0xffffffff);
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < total; x += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = x / (2 * pieces);
    const int64_t r = x - i * 2 * pieces;
    const int tensor = r >= pieces;                       // 0 = K, 1 = V
    const int64_t piece = r - tensor * pieces;
    const uint32_t id = (uint32_t)a.ids[i];
    if (id >= nb) continue;                               // out of the pool: never dereferenced
    char* dev = reinterpret_cast<char*>(tensor ? a.v_pool : a.k_pool) + (int64_t)id * a.page_bytes + piece * 16;
    char* host = reinterpret_cast<char*>(a.host) + x * 16;
    if (a.to_host) {
      *reinterpret_cast<u32x4*>(host) = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(dev));
    } else {
      __builtin_nontemporal_store(*reinterpret_cast<const u32x4*>(host), reinterpret_cast<u32x4*>(dev));
    }
  }
}

}  // namespace

hipError_t launch_copy_blocks(const CopyArgs& a, int grid, hipStream_t stream) {
  hipLaunchKernelGGL(copy_blocks_kernel, dim3(grid), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace kvt
