// Append (writeback) of the new tokens' K/V into their cache pages.
//
// The KV of newly prefilled tokens becomes reusable once written into the
// pages the sequence's block table names (paper §5.1: KV exists only for
// tokens that took part in inference; §6.2: writeback after prefill).  The
// operation is a pure byte copy, so the kernel is an HBM-bound scatter:
// every thread moves 16-byte pieces; a wave covers 1 KiB of consecutive
// source bytes (four token-head rows), and each 256-byte row (bf16, D=128)
// lands contiguously in its page slot.
#include "kvt_internal.h"

namespace kvt {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Index of the launch-local sequence that owns packed row r (rows are in
// sequence order; row_off is non-decreasing).
__device__ inline int find_seq(const AppendArgs& a, int32_t row) {
  int lo = 0, hi = a.nseq - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (a.seq[mid].row_off <= row) lo = mid; else hi = mid - 1;
  }
  return lo;
}

template <int ELEM_BYTES, int D>
__global__ __launch_bounds__(256) void append_kv_kernel(AppendArgs a) {
  constexpr int kPieces = D * ELEM_BYTES / 16;   // 16-byte pieces per (token, head) row
  const int hkv = a.num_kv_heads;
  const int64_t per_row = (int64_t)hkv * kPieces;
  const int64_t total = (int64_t)a.rows * per_row;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const u32x4* kn = reinterpret_cast<const u32x4*>(a.k_new);
  const u32x4* vn = reinterpret_cast<const u32x4*>(a.v_new);
  u32x4* kp = reinterpret_cast<u32x4*>(a.k_pool);
  u32x4* vp = reinterpret_cast<u32x4*>(a.v_pool);
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += stride) {
    const int32_t r = (int32_t)(idx / per_row);            // launch-local row
    const int32_t rem = (int32_t)(idx - (int64_t)r * per_row);
    const int32_t g = rem / kPieces;
    const int32_t c = rem - g * kPieces;
    const int32_t row = a.row_begin + r;                   // packed row of the call
    const SeqDesc sd = a.seq[find_seq(a, row)];
    const int32_t pos = sd.prefix + (row - sd.row_off);    // logical position
    const int32_t bid = a.block_table[(int64_t)sd.seq * a.max_blocks + pos / kBlock];
    if ((uint64_t)(uint32_t)bid >= (uint64_t)a.num_blocks || bid < 0) continue;
    const int64_t dst = ((((int64_t)bid * hkv + g) * kBlock) + (pos % kBlock)) * kPieces + c;
    const int64_t src = ((int64_t)row * hkv + g) * kPieces + c;
    const u32x4 kv = __builtin_nontemporal_load(kn + src);
    const u32x4 vv = __builtin_nontemporal_load(vn + src);
    kp[dst] = kv;
    vp[dst] = vv;
  }
}

}  // namespace

hipError_t launch_append(const AppendArgs& a, int dtype, int head_dim, hipStream_t stream) {
  const int elem = dtype == 0 ? 2 : 4;
  const int64_t pieces = (int64_t)a.rows * a.num_kv_heads * head_dim * elem / 16;
  int64_t blocks = (pieces + 255) / 256;
  if (blocks > 8192) blocks = 8192;   // grid-stride beyond 32 resident workgroups per CU
  if (blocks < 1) blocks = 1;
  dim3 grid((unsigned)blocks), block(256);
  if (dtype == 0 && head_dim == 128) hipLaunchKernelGGL((append_kv_kernel<2, 128>), grid, block, 0, stream, a);
  else if (dtype == 0 && head_dim == 64) hipLaunchKernelGGL((append_kv_kernel<2, 64>), grid, block, 0, stream, a);
  else if (dtype == 1 && head_dim == 128) hipLaunchKernelGGL((append_kv_kernel<4, 128>), grid, block, 0, stream, a);
  else hipLaunchKernelGGL((append_kv_kernel<4, 64>), grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace kvt
