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

typedef __attribute__((address_space(3))) __bf16 lds_bf16;

// One K/V tile of 64 keys in LDS: [K|V][key][D] bf16, 16-byte chunks of each
// key row XOR-swizzled.  Two tiles form the double buffer; they are distinct
// objects so the compiler can tell loads into one from reads of the other.
template <int D>
struct KvTile {
  __bf16 kv[2 * kExtKeysPerTile * D];
};

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void extend_fwd_kernel(const ExtendArgs a) {
  constexpr int KT = kExtKeysPerTile;            // 64 keys per tile = 4 pages
  constexpr int CHUNKS = D / 8;                  // 16-byte chunks per key row
  constexpr int ROWB = D * 2;                    // bytes per key row in LDS
  constexpr int RPR = 1024 / ROWB;               // key rows per 1 KiB wave load
  constexpr int NREG = KT * ROWB / 1024 / kExtWaves;  // 1 KiB loads per wave per tensor
  constexpr int KSTEPS = D / 16;                 // MFMA k-steps of the score product
  constexpr int DT = D / 32;                     // 32-wide output column tiles
  constexpr int TILE_ELEMS = KT * D;
  constexpr bool kDirect = sizeof(T) == 2;       // bf16 storage: global -> LDS directly
  constexpr float kRescaleSlack = 8.0f;          // log2 headroom before O is rescaled
  __shared__ __attribute__((aligned(1024))) KvTile<D> tile0;
  __shared__ __attribute__((aligned(1024))) KvTile<D> tile1;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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
  const int nblk = (L + kBlock - 1) / kBlock;

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
  // the block table is read-only here: a constant-address-space view lets
  // wave-uniform page lookups become scalar loads
  const __attribute__((address_space(4))) int32_t* bt =
      (const __attribute__((address_space(4))) int32_t*)(a.block_table + (int64_t)sd.seq * a.max_blocks);
  const uint32_t nb_max = (uint32_t)min<int64_t>(a.num_blocks, 0x7fffffff) - 1u;

  // ---- gather geometry: wave `wave`, load i covers key rows RPR*(wave+8i) ..
  // +RPR-1 of the tile, all inside one page.  Lane l lands at LDS byte
  // 16*l of that 1 KiB run, i.e. row RPR*(wave+8i) + l/CHUNKS, physical chunk
  // l%CHUNKS, so it fetches logical chunk (l%CHUNKS) ^ swizzle(row).
  int keyrow[NREG], lds_off[NREG], chunk_off[NREG], page_in_tile[NREG];
#pragma unroll
  for (int i = 0; i < NREG; ++i) {
    const int run = wave + kExtWaves * i;
    keyrow[i] = RPR * run + lane / CHUNKS;
    page_in_tile[i] = (RPR * run) / kBlock;
    lds_off[i] = run * 512;                                   // elements
    chunk_off[i] = (((lane % CHUNKS) ^ swz<D>(keyrow[i])) << 3);
  }
  // physical page ids of the pages a tile needs (wave-uniform, clamped into the pool)
  auto page_ids = [&](int jn, uint32_t (&ids)[NREG]) {
#pragma unroll
    for (int i = 0; i < NREG; ++i) {
      const int page = __builtin_amdgcn_readfirstlane(min(jn * 4 + page_in_tile[i], nblk - 1));
      const uint32_t raw = (uint32_t)bt[page];
      ids[i] = __builtin_amdgcn_readfirstlane(raw > nb_max ? nb_max : raw);
    }
  };
  // element offset of this lane's chunk; positions past the end of the
  // sequence read the last real position instead (finite data whose weight is 0)
  auto src_off = [&](int jn, int i, uint32_t id) -> int64_t {
    const int page = min(jn * 4 + page_in_tile[i], nblk - 1);
    const int last = L - 1 - page * kBlock;
    const int slot = min(keyrow[i] & (kBlock - 1), last);
    return ((((int64_t)id * hkv + g) << 4) + slot) * D + chunk_off[i];
  };
  u32x4 stK[NREG], stV[NREG];   // register staging (fp32 storage only)
  auto issue = [&](int jn, const uint32_t (&ids)[NREG], KvTile<D>& dst) {
#pragma unroll
    for (int i = 0; i < NREG; ++i) {
      const int64_t off = src_off(jn, i, ids[i]);
      if constexpr (kDirect) {
        lds_bf16* kd = (lds_bf16*)dst.kv + lds_off[i];
        __builtin_amdgcn_global_load_lds((const void*)(kpool + off), (__attribute__((address_space(3))) void*)kd, 16, 0, 0);
        __builtin_amdgcn_global_load_lds((const void*)(vpool + off), (__attribute__((address_space(3))) void*)(kd + TILE_ELEMS), 16, 0, 0);
      } else {
        stK[i] = load8(kpool + off);
        stV[i] = load8(vpool + off);
      }
    }
  };
  auto stash = [&](KvTile<D>& dst) {
    if constexpr (!kDirect) {
#pragma unroll
      for (int i = 0; i < NREG; ++i) {
        *reinterpret_cast<u32x4*>(dst.kv + lds_off[i] + lane * 8) = stK[i];
        *reinterpret_cast<u32x4*>(dst.kv + TILE_ELEMS + lds_off[i] + lane * 8) = stV[i];
      }
    }
  };

  f32x16 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = (f32x16){};
  float m_ref = -INFINITY;   // reference max of scale*log2e*score (may trail the true max by < 8)
  float l_run = 0.f;         // this lane's share of sum 2^(s*c - m_ref)
  const float c = a.scale_log2;
  const int g16 = (lane >> 4) & 1;
  const int rsel = (lane & 15) >> 2;

  auto compute = [&](int j, const KvTile<D>& tl) {
    const __bf16* ks = tl.kv;
    const __bf16* vs = tl.kv + TILE_ELEMS;
    // ---- S^T = K Q^T, two independent 32-key chains interleaved
    f32x16 s[2] = {{}, {}};
    const int sw0 = swz<D>(l32), sw1 = swz<D>(32 + l32);
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) {
      const int cl = 2 * kk + hh;
      const bf16x8 k0 = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(ks + l32 * D + ((cl ^ sw0) << 3)));
      const bf16x8 k1 = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(ks + (32 + l32) * D + ((cl ^ sw1) << 3)));
      s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, qreg[kk], s[0], 0, 0, 0);
      s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, qreg[kk], s[1], 0, 0, 0);
    }
    // ---- causal mask: only tiles that reach past the tile's first query
    if (j * KT + KT - 1 > lim_min) {
#pragma unroll
      for (int half = 0; half < 2; ++half)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int kabs = j * KT + half * 32 + 8 * (e >> 2) + 4 * hh + (e & 3);
          if (kabs > lim) s[half][e] = -INFINITY;
        }
    }
    // ---- online softmax (log2 domain); O and l are rescaled only when the
    // tile max passes the reference by more than the slack
    float mx = -INFINITY;
#pragma unroll
    for (int half = 0; half < 2; ++half)
#pragma unroll
      for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[half][e]);
    const float mxc = pair_max(mx) * c;
    const bool up = mxc > m_ref + kRescaleSlack;
    if (__builtin_amdgcn_ballot_w64(up) != 0) {
      const float m_new = up ? mxc : m_ref;
      const float alpha = __builtin_amdgcn_exp2f(m_ref - m_new);   // 1 where unchanged, 0 from -inf
      m_ref = m_new;
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
    }
    const float m_use = (m_ref == -INFINITY) ? 0.f : m_ref;
    float rs = 0.f;
#pragma unroll
    for (int half = 0; half < 2; ++half)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[half][e], c, -m_use));
        s[half][e] = p;
        rs += p;
      }
    l_run += rs;
    // ---- P^T as the B operand: key group kg = 16 keys = 8 accumulators
    bf16x8 pb[4];
#pragma unroll
    for (int kg = 0; kg < 4; ++kg) {
      const f32x16& sv = s[kg >> 1];
      const int b0 = (kg & 1) * 8;
      u32x4 wv;
#pragma unroll
      for (int q2 = 0; q2 < 4; ++q2)
        wv[q2] = __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){sv[b0 + 2 * q2], sv[b0 + 2 * q2 + 1]}, bf16x2));
      pb[kg] = __builtin_bit_cast(bf16x8, wv);
    }
    // ---- O^T += V^T P^T; V^T from the row-major tile by transposed reads
    const lds_bf16* vl = (const lds_bf16*)vs;
#pragma unroll
    for (int kg = 0; kg < 4; ++kg) {
      const int key1 = kg * 16 + 4 * hh + rsel;
      const int key2 = key1 + 8;
      const int sw1k = swz<D>(key1), sw2k = swz<D>(key2);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int dcol = dt * 32 + g16 * 16 + 4 * (lane & 3);
        const int o1 = key1 * D + (((dcol >> 3) ^ sw1k) << 3) + (dcol & 7);
        const int o2 = key2 * D + (((dcol >> 3) ^ sw2k) << 3) + (dcol & 7);
        const bf16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vl + o1));
        const bf16x4 v2 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vl + o2));
        const bf16x8 vf = __builtin_shufflevector(v1, v2, 0, 1, 2, 3, 4, 5, 6, 7);
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[kg], o[dt], 0, 0, 0);
      }
    }
  };

  // ---- pipeline: tile j is computed from one buffer while tile j+1 streams
  // into the other; page ids run two tiles ahead.
  uint32_t ids[NREG];
  page_ids(j0, ids);
  if (j0 < j1) {
    issue(j0, ids, tile0);
    stash(tile0);
  }
  page_ids(j0 + 1, ids);
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
  __syncthreads();
  for (int j = j0; j < j1; j += 2) {
    if (j + 1 < j1) {
      issue(j + 1, ids, tile1);
      page_ids(j + 2, ids);
    }
    compute(j, tile0);
    if (j + 1 < j1) stash(tile1);
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();
    if (j + 1 >= j1) break;
    if (j + 2 < j1) {
      issue(j + 2, ids, tile0);
      page_ids(j + 3, ids);
    }
    compute(j + 1, tile1);
    if (j + 2 < j1) stash(tile0);
    __builtin_amdgcn_s_waitcnt(0x0F70);
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
    if (a.lse != nullptr && hh == 0) a.lse[qrow] = (m_ref + __builtin_log2f(l_tot)) * kLn2;
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
      a.part_ml[prow * 2] = m_ref;
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
