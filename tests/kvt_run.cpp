// Test driver: a native caller of the C ABI -- no Python, no torch.  Reads
// one batch from a binary file, runs kvt_append_kv then kvt_extend_attention
// on the HIP device, and writes out and lse (tests/test_gpu_native.py checks
// them against the oracle).  Built by the package build next to this file.
//
//   kvt_run <input file> <output file>
//
// Input: int32 B, Hq, Hkv, D, num_blocks, max_blocks; float32 scale; int32
// prefix_len[B], suffix_len[B], block_table[B][max_blocks]; then bf16 (raw
// 16-bit) k_pool and v_pool [num_blocks][Hkv][16][D], k_new and v_new
// [T][Hkv][D], q [T][Hq][D] with T = sum of suffix_len.
// Output: bf16 out [T][Hq][D], then float32 lse [T][Hq].
// Exit status: 0 on success, 1 on a bad file, 2 on a HIP error, 3 on a
// library error (its status string is printed).
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstdio>
#include <vector>

#include "kvt.h"

namespace {

template <typename T>
bool read_vec(FILE* f, std::vector<T>& v, size_t n) {
  v.resize(n);
  return fread(v.data(), sizeof(T), n, f) == n;
}

bool hip_ok(hipError_t e, const char* what) {
  if (e == hipSuccess) return true;
  std::fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
  return false;
}

// device buffer of `bytes`, filled from src unless src is NULL
void* to_device(const void* src, size_t bytes) {
  void* p = nullptr;
  if (!hip_ok(hipMalloc(&p, bytes ? bytes : 1), "hipMalloc")) return nullptr;
  if (src != nullptr && bytes && !hip_ok(hipMemcpy(p, src, bytes, hipMemcpyHostToDevice), "hipMemcpy")) return nullptr;
  return p;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 3) {
    std::fprintf(stderr, "usage: %s <input> <output>\n", argv[0]);
    return 1;
  }
  FILE* f = std::fopen(argv[1], "rb");
  if (f == nullptr) return 1;
  int32_t hdr[6];
  float scale = 0.f;
  if (fread(hdr, sizeof(int32_t), 6, f) != 6 || fread(&scale, sizeof(float), 1, f) != 1) return 1;
  const int32_t B = hdr[0], Hq = hdr[1], Hkv = hdr[2], D = hdr[3], NB = hdr[4], MB = hdr[5];
  if (B < 1 || Hq < 1 || Hkv < 1 || D < 1 || NB < 1 || MB < 1) return 1;
  std::vector<int32_t> P, S, table;
  if (!read_vec(f, P, B) || !read_vec(f, S, B) || !read_vec(f, table, (size_t)B * MB)) return 1;
  int64_t T = 0;
  for (int b = 0; b < B; ++b) T += S[b];
  const size_t pool_elems = (size_t)NB * Hkv * 16 * D;
  std::vector<uint16_t> kp, vp, kn, vn, q;
  if (!read_vec(f, kp, pool_elems) || !read_vec(f, vp, pool_elems) || !read_vec(f, kn, (size_t)T * Hkv * D) ||
      !read_vec(f, vn, (size_t)T * Hkv * D) || !read_vec(f, q, (size_t)T * Hq * D))
    return 1;
  std::fclose(f);

  void* dk = to_device(kp.data(), kp.size() * 2);
  void* dv = to_device(vp.data(), vp.size() * 2);
  void* dkn = to_device(kn.data(), kn.size() * 2);
  void* dvn = to_device(vn.data(), vn.size() * 2);
  void* dq = to_device(q.data(), q.size() * 2);
  void* dt = to_device(table.data(), table.size() * 4);
  void* dout = to_device(nullptr, (size_t)T * Hq * D * 2);
  void* dlse = to_device(nullptr, (size_t)T * Hq * 4);
  if (!dk || !dv || !dkn || !dvn || !dq || !dt || !dout || !dlse) return 2;
  hipStream_t stream;
  if (!hip_ok(hipStreamCreate(&stream), "hipStreamCreate")) return 2;

  kvt_pool pool = {dk, dv, NB, Hkv, D, KVT_DTYPE_BF16};
  kvt_seqs seqs = {B, P.data(), S.data(), (const int32_t*)dt, table.data(), MB};   // checked mode
  kvt_status st = kvt_append_kv(&pool, &seqs, dkn, dvn, stream);
  if (st != KVT_OK) {
    std::fprintf(stderr, "kvt_append_kv: %s\n", kvt_status_str(st));
    return 3;
  }
  const size_t ws_bytes = kvt_extend_workspace_bytes(&pool, &seqs, Hq);
  void* ws = nullptr;
  if (ws_bytes && !hip_ok(hipMalloc(&ws, ws_bytes), "hipMalloc")) return 2;
  st = kvt_extend_attention(&pool, &seqs, dq, Hq, scale, dout, (float*)dlse, ws, ws_bytes, stream);
  if (st != KVT_OK) {
    std::fprintf(stderr, "kvt_extend_attention: %s\n", kvt_status_str(st));
    return 3;
  }
  if (!hip_ok(hipStreamSynchronize(stream), "hipStreamSynchronize")) return 2;

  std::vector<uint16_t> out((size_t)T * Hq * D);
  std::vector<float> lse((size_t)T * Hq);
  if (!hip_ok(hipMemcpy(out.data(), dout, out.size() * 2, hipMemcpyDeviceToHost), "hipMemcpy") ||
      !hip_ok(hipMemcpy(lse.data(), dlse, lse.size() * 4, hipMemcpyDeviceToHost), "hipMemcpy"))
    return 2;
  FILE* o = std::fopen(argv[2], "wb");
  if (o == nullptr) return 1;
  fwrite(out.data(), 2, out.size(), o);
  fwrite(lse.data(), 4, lse.size(), o);
  std::fclose(o);
  for (void* p : {dk, dv, dkn, dvn, dq, dt, dout, dlse, ws}) (void)hipFree(p);
  (void)hipStreamDestroy(stream);
  std::printf("kvt_run: %lld tokens, workspace %zu bytes\n", (long long)T, ws_bytes);
  return 0;
}
