// Extend attention over a paged KV cache, gfx950.
//
// The S_b new tokens of sequence b attend causally over the P_b reused
// positions plus themselves (prefix reuse in place of re-prefill, paper §1,
// §2.2).  Work decomposition, per workgroup:
//   * one kv-head g and 256 packed query rows (row r = token r/G, head
//     g*G + r%G): the G query heads that share a kv-head share every K/V
//     tile staged in LDS;
//   * 8 waves, each owning 32 rows; the wave computes S^T = K Q^T with
//     v_mfma_f32_32x32x16_bf16 (keys on the MFMA rows, queries on the
//     columns), so a query's scores sit in one lane pair (l, l+32) and the
//     row max / row sum need a single permlane32 swap;
//   * the probabilities leave the S^T accumulators already in the B-operand
//     layout of O^T += V^T P^T; the V^T operand comes straight from the
//     row-major V tile through ds_read_b64_tr_b16;
//   * fp32 online softmax in log2 units (scale*log2e folded into one FMA);
//   * K/V tiles of 64 keys (4 pages) are gathered through the block table
//     into a double-buffered LDS ring; every page contributes one contiguous
//     run of 16*D elements per kv-head, read with 16-byte coalesced loads.
// Positions past the end of the sequence and unused page slots are never
// multiplied in: their K/V are replaced by zeros in LDS and their scores by
// -inf.
#include "kvt_internal.h"

namespace kvt {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr float kLn2 = 0.693147180559945309f;
constexpr int kThreads = kExtWaves * 64;

// XOR swizzle of the 16-byte chunks of one key row in LDS.  Over any 8
// consecutive keys the K-operand reads (one chunk column, 8 rows) hit 8
// distinct bank groups, and over any 4 consecutive keys the transposed V
// reads (two adjacent chunks, 4 rows) do too.
template <int D>
__device__ __forceinline__ int swz(int key) {
  const int s = ((key & 3) << 1) | ((key >> 2) & 1) | (((key >> 3) & 1) << 3);
  return D == 128 ? s : (s & 7);
}

// 8 consecutive elements as bf16 (fp32 storage is rounded to nearest even).
__device__ __forceinline__ u32x4 load8(const __bf16* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
__device__ __forceinline__ u32x4 load8(const float* p) {
  const f32x4 a = *reinterpret_cast<const f32x4*>(p);
  const f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
  u32x4 r;
  r[0] = __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){a[0], a[1]}, bf16x2));
  r[1] = __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){a[2], a[3]}, bf16x2));
  r[2] = __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){b[0], b[1]}, bf16x2));
  r[3] = __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){b[2], b[3]}, bf16x2));
  return r;
}

__device__ __forceinline__ void store4(__bf16* p, float a, float b, float c, float d) {
  u32x2 v;
  v[0] = __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){a, b}, bf16x2));
  v[1] = __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){c, d}, bf16x2));
  *reinterpret_cast<u32x2*>(p) = v;
}
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<f32x4*>(p) = (f32x4){a, b, c, d};
}

// Own value and the partner lane's (l ^ 32) value, via v_permlane32_swap:
// with vdst = vsrc = x the swap leaves {x_lo, x_lo} in vdst and {x_hi, x_hi}
// in vsrc, so every lane sees both halves' values in the two results.  The
// two results are copied into scalars before the bit cast: a bit cast applied
// directly to an element of the returned vector reads element 0 for both.
__device__ __forceinline__ void pair_values(float x, float& a, float& b) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto p = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const unsigned p0 = p[0];
  const unsigned p1 = p[1];
  a = __builtin_bit_cast(float, p0);
  b = __builtin_bit_cast(float, p1);
}
__device__ __forceinline__ float pair_max(float x) {
  float a, b;
  pair_values(x, a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float pair_sum(float x) {
  float a, b;
  pair_values(x, a, b);
  return a + b;
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void extend_fwd_kernel(const ExtendArgs a) {
  constexpr int KT = kExtKeysPerTile;            // 64 keys per tile
  constexpr int CHUNKS = D / 8;                  // 16-byte chunks per key row
  constexpr int PIECES = KT * CHUNKS / kThreads; // chunks per thread per tensor per tile
  constexpr int KSTEPS = D / 16;                 // MFMA k-steps of the score product
  constexpr int DT = D / 32;                     // 32-wide output column tiles
  constexpr int TILE_ELEMS = KT * D;
  __shared__ __attribute__((aligned(16))) __bf16 smem[2 * 2 * TILE_ELEMS];  // [buf][K|V][key][D]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int hh = lane >> 5;     // lane half
  const int l32 = lane & 31;

  // ---- which (sequence, kv-head, row tile, key split) this workgroup owns
  const int hkv = a.num_kv_heads;
  const int g = blockIdx.x % hkv;
  const int unit = blockIdx.x / hkv;
  int si = 0;
  while (si + 1 < a.nseq && a.unit_begin[si + 1] <= unit) ++si;
  const SeqDesc sd = a.seq[si];
  const int local = unit - a.unit_begin[si];
  const int G = a.group;
  const int rows_seq = sd.suffix * G;
  const int ntile = (rows_seq + kExtTileRows - 1) / kExtTileRows;
  const int rt = ntile - 1 - local / a.nsplit;   // longest row tile first
  const int split = local % a.nsplit;
  const int r0 = rt * kExtTileRows;
  const int P = sd.prefix;
  const int L = P + sd.suffix;

  // keys this tile needs: up to the last query's own position
  const int t_last = min(sd.suffix - 1, (r0 + kExtTileRows - 1) / G);
  const int kmax = P + t_last + 1;
  const int ntiles_kv = (kmax + KT - 1) / KT;
  const int per_split = (ntiles_kv + a.nsplit - 1) / a.nsplit;
  const int j0 = split * per_split;
  const int j1 = min(ntiles_kv, j0 + per_split);
  const int lim_min = P + r0 / G;   // smallest causal limit of the tile

  // ---- this lane's query row
  int r = r0 + wave * kExtRowsPerWave + l32;
  const bool row_valid = r < rows_seq;
  if (!row_valid) r = rows_seq - 1;
  const int t = r / G;
  const int h = g * G + (r - t * G);
  const int lim = P + t;                               // last visible position
  const int64_t qrow = (int64_t)(sd.row_off + t) * a.num_q_heads + h;

  const T* qp = reinterpret_cast<const T*>(a.q) + qrow * D;
  bf16x8 qreg[KSTEPS];
#pragma unroll
  for (int kk = 0; kk < KSTEPS; ++kk) qreg[kk] = __builtin_bit_cast(bf16x8, load8(qp + kk * 16 + hh * 8));

  const T* kpool = reinterpret_cast<const T*>(a.k_pool);
  const T* vpool = reinterpret_cast<const T*>(a.v_pool);
  const int32_t* bt = a.block_table + (int64_t)sd.seq * a.max_blocks;

  // ---- global -> register staging of one K/V tile
  u32x4 stK[PIECES], stV[PIECES];
  auto fetch = [&](int j) {
#pragma unroll
    for (int i = 0; i < PIECES; ++i) {
      const int p = tid + i * kThreads;
      const int key = p / CHUNKS;
      const int cl = p % CHUNKS;
      const int kabs = j * KT + key;
      u32x4 kv = {0u, 0u, 0u, 0u}, vv = {0u, 0u, 0u, 0u};
      if (kabs < L) {
        const int bid = bt[kabs / kBlock];
        if (bid >= 0 && (int64_t)bid < a.num_blocks) {
          const int64_t off = ((((int64_t)bid * hkv + g) * kBlock) + (kabs % kBlock)) * D + cl * 8;
          kv = load8(kpool + off);
          vv = load8(vpool + off);
        }
      }
      stK[i] = kv;
      stV[i] = vv;
    }
  };
  auto stash = [&](int buf) {
    __bf16* ks = smem + buf * 2 * TILE_ELEMS;
    __bf16* vs = ks + TILE_ELEMS;
#pragma unroll
    for (int i = 0; i < PIECES; ++i) {
      const int p = tid + i * kThreads;
      const int key = p / CHUNKS;
      const int cl = p % CHUNKS;
      const int o = key * D + ((cl ^ swz<D>(key)) << 3);
      *reinterpret_cast<u32x4*>(ks + o) = stK[i];
      *reinterpret_cast<u32x4*>(vs + o) = stV[i];
    }
  };

  f32x16 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = (f32x16){};
  float m_run = -INFINITY;   // running max of scale*log2e*score
  float l_run = 0.f;         // this lane's share of the running row sum
  const float c = a.scale_log2;

  if (j0 < j1) {
    fetch(j0);
    stash(0);
  }
  __syncthreads();

  for (int j = j0; j < j1; ++j) {
    const int buf = (j - j0) & 1;
    if (j + 1 < j1) fetch(j + 1);
    const __bf16* ks = smem + buf * 2 * TILE_ELEMS;
    const __bf16* vs = ks + TILE_ELEMS;

    // ---- S^T = K Q^T for two 32-key halves
    f32x16 s[2];
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int key = half * 32 + l32;
      const __bf16* krow = ks + key * D;
      const int sw = swz<D>(key);
      f32x16 acc = {};
#pragma unroll
      for (int kk = 0; kk < KSTEPS; ++kk) {
        const int cl = 2 * kk + hh;
        const bf16x8 kf = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(krow + ((cl ^ sw) << 3)));
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qreg[kk], acc, 0, 0, 0);
      }
      s[half] = acc;
    }

    // ---- causal mask (only tiles that reach past the tile's first query)
    if (j * KT + KT - 1 > lim_min) {
#pragma unroll
      for (int half = 0; half < 2; ++half)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int kabs = j * KT + half * 32 + 8 * (e >> 2) + 4 * hh + (e & 3);
          if (kabs > lim) s[half][e] = -INFINITY;
        }
    }

    // ---- online softmax (log2 domain)
    float mx = -INFINITY;
#pragma unroll
    for (int half = 0; half < 2; ++half)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[half][e]);
    mx = pair_max(mx);
    const float m_new = fmaxf(m_run, mx * c);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
    m_run = m_new;
    float rs = 0.f;
#pragma unroll
    for (int half = 0; half < 2; ++half)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[half][e], c, -m_use));
        s[half][e] = p;
        rs += p;
      }
    l_run = l_run * alpha + rs;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;

    // ---- P^T as the B operand: key group kg = 16 keys = 8 accumulators
    bf16x8 pb[4];
#pragma unroll
    for (int kg = 0; kg < 4; ++kg) {
      const f32x16& sv = s[kg >> 1];
      const int b0 = (kg & 1) * 8;
      u32x4 w;
#pragma unroll
      for (int q2 = 0; q2 < 4; ++q2)
        w[q2] = __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){sv[b0 + 2 * q2], sv[b0 + 2 * q2 + 1]}, bf16x2));
      pb[kg] = __builtin_bit_cast(bf16x8, w);
    }

    // ---- O^T += V^T P^T; V^T from the row-major tile by transposed reads
    const int g16 = (lane >> 4) & 1;
    const int rsel = (lane & 15) >> 2;
#pragma unroll
    for (int kg = 0; kg < 4; ++kg) {
      const int key1 = kg * 16 + 4 * hh + rsel;
      const int key2 = key1 + 8;
      const int sw1 = swz<D>(key1), sw2 = swz<D>(key2);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int dcol = dt * 32 + g16 * 16 + 4 * (lane & 3);
        const int o1 = key1 * D + (((dcol >> 3) ^ sw1) << 3) + (dcol & 7);
        const int o2 = key2 * D + (((dcol >> 3) ^ sw2) << 3) + (dcol & 7);
        const bf16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)((__attribute__((address_space(3))) __bf16*)smem + (vs - smem) + o1));
        const bf16x4 v2 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)((__attribute__((address_space(3))) __bf16*)smem + (vs - smem) + o2));
        const bf16x8 vf = __builtin_shufflevector(v1, v2, 0, 1, 2, 3, 4, 5, 6, 7);
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[kg], o[dt], 0, 0, 0);
      }
    }

    if (j + 1 < j1) stash(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue
  const float l_tot = pair_sum(l_run);
  if (!row_valid) return;
  if (a.nsplit == 1) {
    const float inv = 1.0f / l_tot;
    T* op = reinterpret_cast<T*>(a.out) + qrow * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = dt * 32 + 8 * i + 4 * hh;
        store4(op + d, o[dt][4 * i] * inv, o[dt][4 * i + 1] * inv, o[dt][4 * i + 2] * inv, o[dt][4 * i + 3] * inv);
      }
    if (a.lse != nullptr && hh == 0) a.lse[qrow] = (m_run + __builtin_log2f(l_tot)) * kLn2;
  } else {
    const int64_t prow = (int64_t)split * a.total_rows * a.num_q_heads + qrow;
    float* op = a.part_o + prow * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = dt * 32 + 8 * i + 4 * hh;
        store4(op + d, o[dt][4 * i], o[dt][4 * i + 1], o[dt][4 * i + 2], o[dt][4 * i + 3]);
      }
    if (hh == 0) {
      a.part_ml[prow * 2] = m_run;
      a.part_ml[prow * 2 + 1] = l_tot;
    }
  }
}

// Merge the per-split partial results of each row (fixed split order):
//   m* = max_s m_s,  w_s = 2^(m_s - m*),  out = sum_s w_s O_s / sum_s w_s l_s.
template <typename T, int D>
__global__ __launch_bounds__(256) void extend_combine_kernel(const CombineArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // (row, 4-column group)
  constexpr int Q4 = D / 4;
  if (idx >= a.rows * Q4) return;
  const int64_t row = idx / Q4;
  const int c4 = (int)(idx - row * Q4) * 4;
  float mstar = -INFINITY;
  for (int s = 0; s < a.nsplit; ++s) mstar = fmaxf(mstar, a.part_ml[(s * a.rows + row) * 2]);
  float lsum = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < a.nsplit; ++s) {
    const int64_t pr = s * a.rows + row;
    const float m = a.part_ml[pr * 2];
    const float w = (m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m - mstar);
    lsum += w * a.part_ml[pr * 2 + 1];
    const f32x4 v = *reinterpret_cast<const f32x4*>(a.part_o + pr * D + c4);
    acc += w * v;
  }
  const float inv = 1.0f / lsum;
  store4(reinterpret_cast<T*>(a.out) + row * D + c4, acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
  if (a.lse != nullptr && c4 == 0) a.lse[row] = (mstar + __builtin_log2f(lsum)) * kLn2;
}

}  // namespace

hipError_t launch_extend(const ExtendArgs& a, int dtype, int head_dim, int grid, hipStream_t stream) {
  dim3 g(grid), b(kThreads);
  if (dtype == 0 && head_dim == 128) hipLaunchKernelGGL((extend_fwd_kernel<__bf16, 128>), g, b, 0, stream, a);
  else if (dtype == 0 && head_dim == 64) hipLaunchKernelGGL((extend_fwd_kernel<__bf16, 64>), g, b, 0, stream, a);
  else if (dtype == 1 && head_dim == 128) hipLaunchKernelGGL((extend_fwd_kernel<float, 128>), g, b, 0, stream, a);
  else hipLaunchKernelGGL((extend_fwd_kernel<float, 64>), g, b, 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_combine(const CombineArgs& a, int dtype, int head_dim, hipStream_t stream) {
  const int64_t n = a.rows * (head_dim / 4);
  dim3 g((unsigned)((n + 255) / 256)), b(256);
  if (dtype == 0 && head_dim == 128) hipLaunchKernelGGL((extend_combine_kernel<__bf16, 128>), g, b, 0, stream, a);
  else if (dtype == 0 && head_dim == 64) hipLaunchKernelGGL((extend_combine_kernel<__bf16, 64>), g, b, 0, stream, a);
  else if (dtype == 1 && head_dim == 128) hipLaunchKernelGGL((extend_combine_kernel<float, 128>), g, b, 0, stream, a);
  else hipLaunchKernelGGL((extend_combine_kernel<float, 64>), g, b, 0, stream, a);
  return hipGetLastError();
}

}  // namespace kvt
