// Launch descriptors shared by the host dispatcher (kvt_api.cpp) and the
// device code (kvt_append.hip, kvt_extend.hip).  Per-call sequence metadata
// travels by value in the kernel arguments, so a call needs no device
// allocation and no host-to-device copy; calls with more sequences than one
// descriptor holds are split over several launches.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvt {

constexpr int kBlock = 16;          // tokens per cache page
constexpr int kSeqsPerLaunch = 256;  // sequences described by one launch (about 5.2 KiB of kernel arguments)

// Extend tiling: one workgroup = 8 waves x 32 packed query rows, 64-key tiles.
constexpr int kExtWaves = 8;
constexpr int kExtRowsPerWave = 32;    // one 32-row MFMA block
constexpr int kExtTileRows = kExtWaves * kExtRowsPerWave;   // 256
constexpr int kExtKeysPerTile = 64;
constexpr int kMaxSplits = 16;

// Decode tiling: one workgroup = 4 waves over one (sequence, kv-head, key
// split); each wave streams its own 32-key tiles; up to 32 query rows (G).
constexpr int kDecWaves = 4;
constexpr int kDecKeysPerTile = 32;
constexpr int kDecMaxGroup = 32;

struct SeqDesc {
  int32_t seq;      // row of the block table
  int32_t prefix;   // P_b
  int32_t suffix;   // S_b
  int32_t row_off;  // first packed token row of the sequence (whole call)
};

struct AppendArgs {
  const void* k_new;
  const void* v_new;
  void* k_pool;
  void* v_pool;
  const int32_t* block_table;
  int64_t num_blocks;
  int32_t max_blocks;
  int32_t num_kv_heads;
  int32_t row_begin;  // first packed row covered by this launch
  int32_t rows;       // rows covered by this launch
  int32_t nseq;
  SeqDesc seq[kSeqsPerLaunch];  // in packed-row order
};

struct ExtendArgs {
  const void* q;
  const void* k_pool;
  const void* v_pool;
  void* out;
  float* lse;        // may be null
  float* part_o;     // [nsplit][total_rows * Hq][D] when nsplit > 1
  float* part_ml;    // [nsplit][total_rows * Hq][2]  (running max in log2 units, row sum)
  const int32_t* block_table;
  int64_t num_blocks;
  int32_t max_blocks;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t group;        // Hq / Hkv
  float scale_log2;     // scale * log2(e)
  int32_t kbeg;         // first key position attended (multiple of 16; 0 = from the start)
  int32_t kend;         // key positions >= kend are not attended (INT32_MAX = no cap)
  int32_t direct;       // 1: write out/lse; 0: write partial (part_base + split)
  int32_t part_base;    // first partial slot of this launch
  int32_t nsplit;
  int32_t total_rows;   // T of the whole call
  int32_t nseq;
  // Extend only: sequences second .. nseq-1 form a second group with their
  // own key range, key splits and first partial slot (a cascade launch: the
  // shared part as sequence 0, the private parts after it); second = nseq
  // when the launch has one group.
  int32_t second;
  int32_t kbeg2, kend2, nsplit2, part_base2;
  int32_t unit_begin[kSeqsPerLaunch + 1];  // prefix sums of (row tiles x nsplit), longest first
  SeqDesc seq[kSeqsPerLaunch];
};

// Launch arguments travel by value; larger batches take several launches.
static_assert(sizeof(ExtendArgs) <= 8192 && sizeof(AppendArgs) <= 8192, "kernel argument block too large");

struct CombineArgs {
  const float* part_o;
  const float* part_ml;
  void* out;
  float* lse;
  int64_t rows;    // T * Hq
  int32_t nsplit;
};

struct CopyArgs {
  void* k_pool;
  void* v_pool;
  const int32_t* ids;   // device, n page ids
  int64_t n;
  void* host;           // pinned host buffer [n][K|V][page_bytes], device-accessible
  int64_t page_bytes;   // bytes of one page of one tensor: Hkv * 16 * D * elem
  int64_t num_blocks;
  int32_t to_host;      // 1: pool -> host; 0: host -> pool
};

// Launchers (device code files).  Return the launch status.
hipError_t launch_append(const AppendArgs& a, int dtype, int head_dim, hipStream_t stream);
hipError_t launch_extend(const ExtendArgs& a, int dtype, int head_dim, int grid, hipStream_t stream);
hipError_t launch_combine(const CombineArgs& a, int dtype, int head_dim, hipStream_t stream);
hipError_t launch_copy_blocks(const CopyArgs& a, int grid, hipStream_t stream);
// Decode: ExtendArgs with suffix 1 per sequence and nsplit units per sequence.
hipError_t launch_decode(const ExtendArgs& a, int dtype, int head_dim, int grid, hipStream_t stream);
// Device address of the current GPU's copy of the static scratch
// (KVT_NOALLOC_SCRATCH_BYTES), looked up once per device.
hipError_t noalloc_scratch(void** ptr);

}  // namespace kvt
