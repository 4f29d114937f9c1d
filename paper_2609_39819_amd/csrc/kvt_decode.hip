// Paged decode attention, gfx950: one new token per sequence.
//
// A decode step is the suffix-of-one case of extend attention (the new token
// at position P_b sees keys 0..P_b, its own K/V appended first): every
// sequence contributes G = Hq/Hkv query rows per kv-head, and the cost is
// streaming the sequence's K/V once from HBM.  Work decomposition:
//   * one workgroup per (sequence, kv-head, key split), 4 waves;
//   * wave w takes the split's 32-key tiles w, w+4, w+8, ...: each tile is
//     loaded into registers two tiles ahead of its use and stored into the
//     wave's own LDS slot just before it is needed; the slot is private to
//     the wave, so the loop has no barrier (plain loads into registers
//     stream faster from HBM than LDS-DMA gathers, and keep two tiles per
//     wave in flight);
//   * per tile: S^T = K Q^T and O^T += V^T P^T on one 32-row MFMA block
//     (v_mfma_f32_32x32x16_bf16; rows >= G repeat row G-1 and are dropped),
//     with the online softmax of the extend kernel (lazy reference max);
//   * at the end the four waves' (m, l, O) merge through LDS, and the merged
//     row is either the output or, when the key range is split over
//     workgroups, a partial for the split combine.
#include "kvt_device.h"
#include "kvt_internal.h"

namespace kvt {
namespace {

using namespace dev;

constexpr int kWaves = kDecWaves;
constexpr int kTK = kDecKeysPerTile;   // keys per tile = 2 pages

// One wave's ring slot: its K tile then its V tile, [key][D] bf16 with the
// 16-byte chunks of each key row XOR-swizzled as in the extend kernel.
template <int D>
struct DecSlot {
  __bf16 k[kTK * D];
  __bf16 v[kTK * D];
};

template <typename T, int D>
__global__ __launch_bounds__(kWaves * 64) void decode_kernel(const ExtendArgs a) {
  constexpr int CHUNKS = D / 8;                  // 16-byte chunks per key row
  constexpr int ROWB = D * 2;                    // bytes per key row in LDS
  constexpr int RPR = 1024 / ROWB;               // key rows per 1 KiB wave load
  constexpr int NLD = kTK * ROWB / 1024;         // 1 KiB loads per tensor per tile
  constexpr int KSTEPS = D / 16;
  constexpr int DT = D / 32;
  constexpr float kRescaleSlack = 8.0f;
  __shared__ __attribute__((aligned(1024))) DecSlot<D> ring0[kWaves];   // one slot per wave
  __shared__ float ml[kWaves][32][2];            // per wave and row: m (log2 units), l

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hh = lane >> 5;
  const int l32 = lane & 31;

  // ---- which (sequence, kv-head, key split) this workgroup owns
  const int hkv = a.num_kv_heads;
  const int g = blockIdx.x % hkv;
  const int unit = blockIdx.x / hkv;
  const int si = find_seq(a.unit_begin, a.nseq, unit);
  const SeqDesc sd = a.seq[si];
  const int split = unit - a.unit_begin[si];
  const int G = a.group;
  const int L = sd.prefix + 1;                   // keys 0..P_b
  const int nblk = (L + kBlock - 1) / kBlock;
  const int ntk = (L + kTK - 1) / kTK;
  const int per_split = (ntk + a.nsplit - 1) / a.nsplit;
  const int j0 = split * per_split;
  const int j1 = min(ntk, j0 + per_split);
  const int nt = j1 - j0 > wave ? (j1 - j0 - wave + kWaves - 1) / kWaves : 0;   // this wave's tiles

  // ---- this lane's query row (one 32-row block; rows >= G are padding)
  const int h = g * G + min(l32, G - 1);
  const int64_t qrow = (int64_t)sd.row_off * a.num_q_heads + h;
  bf16x8 qreg[KSTEPS];
  {
    const T* qp = reinterpret_cast<const T*>(a.q) + qrow * D;
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) qreg[kk] = __builtin_bit_cast(bf16x8, load8(qp + kk * 16 + hh * 8));
  }

  const T* kpool = reinterpret_cast<const T*>(a.k_pool);
  const T* vpool = reinterpret_cast<const T*>(a.v_pool);
  const __attribute__((address_space(4))) int32_t* bt =
      (const __attribute__((address_space(4))) int32_t*)(a.block_table + (int64_t)sd.seq * a.max_blocks);
  const uint32_t nb_max = (uint32_t)min<int64_t>(a.num_blocks, 0x7fffffff) - 1u;

  // ---- gather geometry: load i of a tile covers key rows RPR*i .. RPR*i+RPR-1
  // (all in one page); lane l lands at byte 16*l of that 1 KiB run, i.e. row
  // RPR*i + l/CHUNKS, physical chunk l%CHUNKS, logical chunk
  // (l%CHUNKS) ^ swizzle(row)
  int chunk_off[NLD];
#pragma unroll
  for (int i = 0; i < NLD; ++i) chunk_off[i] = ((lane % CHUNKS) ^ swz<D>(RPR * i + lane / CHUNKS)) << 3;
  // page ids of a tile (wave-uniform scalar loads, clamped into the pool)
  auto page_ids = [&](int j, uint32_t (&ids)[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int page = __builtin_amdgcn_readfirstlane(min(j * 2 + p, nblk - 1));
      const uint32_t raw = (uint32_t)bt[page];
      ids[p] = __builtin_amdgcn_readfirstlane(raw > nb_max ? nb_max : raw);
    }
  };
  // one tile's K and V as this lane's 16-byte pieces, in registers
  struct Stage {
    u32x4 k[NLD], v[NLD];
  };
  // positions past the end read the last real position (finite; weight 0)
  auto load_tile = [&](int j, const uint32_t (&ids)[2], Stage& st) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int p = (RPR * i) / kBlock;
      const int page = min(j * 2 + p, nblk - 1);
      const int slot = min((RPR * i + lane / CHUNKS) & (kBlock - 1), L - 1 - page * kBlock);
      const int64_t off = ((((int64_t)ids[p] * hkv + g) << 4) + slot) * D + chunk_off[i];
      if constexpr (sizeof(T) == 2) {   // each page is read once: nontemporal loads
        st.k[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kpool + off));
        st.v[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vpool + off));
      } else {
        st.k[i] = load8(kpool + off);
        st.v[i] = load8(vpool + off);
      }
    }
  };
  auto stash = [&](const Stage& st, DecSlot<D>& dst) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      *reinterpret_cast<u32x4*>(dst.k + i * 512 + lane * 8) = st.k[i];
      *reinterpret_cast<u32x4*>(dst.v + i * 512 + lane * 8) = st.v[i];
    }
  };

  f32x16 o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = (f32x16){};
  float m_ref = -INFINITY, l_run = 0.f;
  const float c = a.scale_log2;
  const int g16 = (lane >> 4) & 1;
  const int rsel = (lane & 15) >> 2;
  int koff[KSTEPS], voff[DT][2];
#pragma unroll
  for (int kk = 0; kk < KSTEPS; ++kk) koff[kk] = l32 * D + (((2 * kk + hh) ^ swz<D>(l32)) << 3);
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int r2 = 0; r2 < 2; ++r2) {
      const int key = 8 * r2 + 4 * hh + rsel;
      const int dcol = dt * 32 + g16 * 16 + 4 * (lane & 3);
      voff[dt][r2] = key * D + (((dcol >> 3) ^ swz<D>(key)) << 3) + (dcol & 7);
    }

  // ---- one 32-key tile starting at key kb: scores, softmax, value product
  auto tile = [&](const DecSlot<D>& sl, int kb) __attribute__((always_inline)) {
    f32x16 s = (f32x16){};
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) {
      const bf16x8 kf = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(sl.k + koff[kk]));
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qreg[kk], s, 0, 0, 0);
    }
    if (kb + kTK > L) {   // the sequence ends inside this tile
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (kb + 8 * (e >> 2) + 4 * hh + (e & 3) >= L) s[e] = -INFINITY;
    }
    float mx = s[0];
#pragma unroll
    for (int e = 1; e < 16; ++e) mx = fmaxf(mx, s[e]);
    const float mxc = pair_max(mx) * c;
    const float m_new = (mxc > m_ref + kRescaleSlack) ? mxc : m_ref;
    const float alpha = (m_new == -INFINITY) ? 1.0f : __builtin_amdgcn_exp2f(m_ref - m_new);
    m_ref = m_new;
    if (__builtin_amdgcn_ballot_w64(alpha != 1.0f) != 0) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
    }
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
    float rs = 0.f;
    bf16x8 pb[2];
#pragma unroll
    for (int kg = 0; kg < 2; ++kg) {
      u32x4 wv;
#pragma unroll
      for (int q2 = 0; q2 < 4; ++q2) {
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kg * 8 + 2 * q2], c, -m_use));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kg * 8 + 2 * q2 + 1], c, -m_use));
        const bf16x2 pp = __builtin_convertvector((f32x2){p0, p1}, bf16x2);
        rs = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, rs, false);
        wv[q2] = __builtin_bit_cast(unsigned, pp);
      }
      pb[kg] = __builtin_bit_cast(bf16x8, wv);
    }
    l_run = l_run * alpha + rs;
    const lds_bf16* vl = (const lds_bf16*)sl.v;
#pragma unroll
    for (int kg = 0; kg < 2; ++kg)
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const bf16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vl + voff[dt][0] + kg * 16 * D));
        const bf16x4 v2 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vl + voff[dt][1] + kg * 16 * D));
        const bf16x8 vf = __builtin_shufflevector(v1, v2, 0, 1, 2, 3, 4, 5, 6, 7);
        o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[kg], o[dt], 0, 0, 0);
      }
  };

  // ---- this wave's tiles j0 + wave + kWaves*i.  Tile i+1 is in registers
  // (possibly still in flight) when step i starts; step i starts loading tile
  // i+2 into the registers tile i left, computes tile i from the slot, then
  // stores tile i+1 into the slot (the wave's LDS operations run in order,
  // so the stores follow the reads of tile i).
  DecSlot<D>& s0 = ring0[wave];
  auto jt = [&](int i) { return j0 + wave + kWaves * i; };
  Stage sa, sb;
  uint32_t ids[2];
  if (nt > 0) {
    page_ids(jt(0), ids);
    load_tile(jt(0), ids, sa);
    if (nt > 1) {
      page_ids(jt(1), ids);
      load_tile(jt(1), ids, sb);
    }
    page_ids(jt(2), ids);
    stash(sa, s0);
  }
  auto step = [&](int i, Stage& nxt, Stage& fill) __attribute__((always_inline)) {
    if (i + 2 < nt) {
      load_tile(jt(i + 2), ids, fill);
      page_ids(jt(i + 3), ids);
    }
    tile(s0, jt(i) * kTK);
    if (i + 1 < nt) stash(nxt, s0);
  };
  for (int i = 0; i < nt; i += 2) {
    step(i, sb, sa);
    if (i + 1 >= nt) break;
    step(i + 1, sa, sb);
  }

  // ---- merge the four waves.  Each wave parks its O (fp32, [row][D]) in
  // its own slot-0 region (its loads have all landed and its reads of the
  // ring precede these writes in LDS order) and (m, l) per row in ml; after
  // the barrier every thread merges columns of the G real rows.
  const float l_tot = pair_sum(l_run);
  float* ow = reinterpret_cast<float*>(&s0);     // 32 x D fp32 = one DecSlot
  static_assert(sizeof(DecSlot<D>) >= 32 * D * sizeof(float), "merge buffer");
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int d = dt * 32 + 8 * i + 4 * hh;
      *reinterpret_cast<f32x4*>(ow + l32 * D + d) = (f32x4){o[dt][4 * i], o[dt][4 * i + 1], o[dt][4 * i + 2], o[dt][4 * i + 3]};
    }
  if (hh == 0) {
    ml[wave][l32][0] = m_ref;
    ml[wave][l32][1] = l_tot;
  }
  __syncthreads();
  for (int idx = tid; idx < G * D; idx += kWaves * 64) {
    const int r = idx / D, d = idx - r * D;
    float mstar = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) mstar = fmaxf(mstar, ml[w][r][0]);
    float lsum = 0.f, acc = 0.f;
    if (mstar != -INFINITY) {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float mw = ml[w][r][0];
        const float wt = (mw == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(mw - mstar);
        lsum += wt * ml[w][r][1];
        acc += wt * reinterpret_cast<const float*>(&ring0[w])[r * D + d];
      }
    }
    const int64_t row = (int64_t)sd.row_off * a.num_q_heads + g * G + r;
    if (a.direct) {
      store1(reinterpret_cast<T*>(a.out) + row * D + d, acc / lsum);
      if (a.lse != nullptr && d == 0) a.lse[row] = (mstar + __builtin_log2f(lsum)) * kLn2;
    } else {
      const int64_t prow = (int64_t)(a.part_base + split) * a.total_rows * a.num_q_heads + row;
      a.part_o[prow * D + d] = acc;
      if (d == 0) {
        a.part_ml[prow * 2] = mstar;
        a.part_ml[prow * 2 + 1] = lsum;
      }
    }
  }
}

}  // namespace

hipError_t launch_decode(const ExtendArgs& a, int dtype, int head_dim, int grid, hipStream_t stream) {
  dim3 g(grid), b(kWaves * 64);
  if (dtype == 0 && head_dim == 128) hipLaunchKernelGGL((decode_kernel<__bf16, 128>), g, b, 0, stream, a);
  else if (dtype == 0 && head_dim == 64) hipLaunchKernelGGL((decode_kernel<__bf16, 64>), g, b, 0, stream, a);
  else if (dtype == 1 && head_dim == 128) hipLaunchKernelGGL((decode_kernel<float, 128>), g, b, 0, stream, a);
  else hipLaunchKernelGGL((decode_kernel<float, 64>), g, b, 0, stream, a);
  return hipGetLastError();
}

}  // namespace kvt
