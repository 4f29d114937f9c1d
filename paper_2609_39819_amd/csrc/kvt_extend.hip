// Extend attention over a paged KV cache, gfx950.
//
// The S_b new tokens of sequence b attend causally over the P_b reused
// positions plus themselves (prefix reuse in place of re-prefill, paper §1,
// §2.2).  Work decomposition, per workgroup:
//   * one kv-head g and 256 packed query rows (row r = token r/G, head
//     g*G + r%G): the G query heads that share a kv-head share every K/V
//     tile staged in LDS;
//   * 8 waves (two per SIMD), each owning 32 rows; the wave computes
//     S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (keys on the MFMA rows,
//     queries on the columns), so a query's scores sit in one lane pair
//     (l, l+32) and the row max / row sum need a single permlane32 swap;
//   * the probabilities leave the S^T accumulators already in the B-operand
//     layout of O^T += V^T P^T; the V^T operand comes straight from the
//     row-major V tile through ds_read_b64_tr_b16;
//   * fp32 online softmax in log2 units (scale*log2e folded into one FMA);
//   * K/V tiles of 64 keys (4 pages) are gathered through the block table
//     straight into a double-buffered LDS ring (global_load_lds_dwordx4);
//     every page contributes one contiguous run of 16*D elements per
//     kv-head, read with 16-byte coalesced loads; the next tile streams in
//     while the current one is computed.
// Positions past the end of the sequence and unused page slots are never
// multiplied in: their loads read the last real position instead (finite
// data) and their scores are replaced by -inf, so their weight is exactly 0.
#include "kvt_device.h"
#include "kvt_internal.h"

namespace kvt {
namespace {

using namespace dev;
constexpr int kThreads = kExtWaves * 64;

// One K or V tile of 64 keys in LDS: [key][D] bf16, the 16-byte chunks of
// each key row XOR-swizzled.  A ring slot is one object holding K then V, so
// every operand read of a slot is a per-lane offset plus an immediate; the
// two slots are distinct objects so the compiler can tell the page gather
// into one slot from the operand reads of the other.
template <int D>
struct HalfTile {
  __bf16 e[kExtKeysPerTile * D];
};
template <int D>
struct Slot {
  HalfTile<D>& k;
  HalfTile<D>& v;
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
  constexpr bool kDirect = sizeof(T) == 2;       // bf16 storage: global -> LDS directly
  constexpr float kRescaleSlack = 8.0f;          // log2 headroom before O is rescaled
  constexpr int NB = kExtRowsPerWave / 32;       // 32-row MFMA blocks per wave
  __shared__ __attribute__((aligned(1024))) HalfTile<D> slot0[2];   // K, V
  __shared__ __attribute__((aligned(1024))) HalfTile<D> slot1[2];
  const Slot<D> tile0{slot0[0], slot0[1]}, tile1{slot1[0], slot1[1]};

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hh = lane >> 5;     // lane half
  const int l32 = lane & 31;

  // ---- which (sequence, kv-head, row tile, key split) this workgroup owns
  const int hkv = a.num_kv_heads;
  const int g = blockIdx.x % hkv;
  const int unit = blockIdx.x / hkv;
  const int si = find_seq(a.unit_begin, a.nseq, unit);
  const SeqDesc sd = a.seq[si];
  const int local = unit - a.unit_begin[si];
  // key range, splits and partial slots of this sequence's group
  const bool grp2 = si >= a.second;
  const int kbeg = grp2 ? a.kbeg2 : a.kbeg;
  const int kend = grp2 ? a.kend2 : a.kend;
  const int nsplit = grp2 ? a.nsplit2 : a.nsplit;
  const int part_base = grp2 ? a.part_base2 : a.part_base;
  const int G = a.group;
  const int rows_seq = sd.suffix * G;
  const int ntile = (rows_seq + kExtTileRows - 1) / kExtTileRows;
  const int rt = ntile - 1 - local / nsplit;   // longest row tile first
  const int split = local % nsplit;
  const int r0 = rt * kExtTileRows;
  const int P = sd.prefix;
  const int L = min(P + sd.suffix, kend);      // positions that can be read
  const int nblk = (L + kBlock - 1) / kBlock;

  // keys this tile needs: from kbeg up to the last query's own position
  // (or kend); the range is split evenly over the key splits
  const int t_last = min(sd.suffix - 1, (r0 + kExtTileRows - 1) / G);
  const int kmax = min(P + t_last + 1, kend);
  const int ntiles_kv = (kmax + KT - 1) / KT;
  const int jlo = kbeg / KT;
  const int per_split = (ntiles_kv - jlo + nsplit - 1) / nsplit;
  const int j0 = jlo + split * per_split;
  const int j1 = min(ntiles_kv, j0 + per_split);
  const int lim_min = min(P + r0 / G, kend - 1);   // smallest last-visible key of the tile

  // ---- this lane's query rows: block b = rows kExtRowsPerWave*wave + 32*b + l32
  int lim[NB];
  bool row_valid[NB];
  int64_t qrow[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    int r = r0 + wave * kExtRowsPerWave + b * 32 + l32;
    row_valid[b] = r < rows_seq;
    if (!row_valid[b]) r = rows_seq - 1;
    const int t = r / G;
    const int h = g * G + (r - t * G);
    lim[b] = min(P + t, kend - 1);                    // last visible position
    qrow[b] = (int64_t)(sd.row_off + t) * a.num_q_heads + h;
  }
  bf16x8 qreg[NB][KSTEPS];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const T* qp = reinterpret_cast<const T*>(a.q) + qrow[b] * D;
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) qreg[b][kk] = __builtin_bit_cast(bf16x8, load8(qp + kk * 16 + hh * 8));
  }

  const T* kpool = reinterpret_cast<const T*>(a.k_pool);
  const T* vpool = reinterpret_cast<const T*>(a.v_pool);
  // the block table is read-only here: a constant-address-space view lets
  // wave-uniform page lookups become scalar loads
  const __attribute__((address_space(4))) int32_t* bt =
      (const __attribute__((address_space(4))) int32_t*)(a.block_table + (int64_t)sd.seq * a.max_blocks);
  const uint32_t nb_max = (uint32_t)min<int64_t>(a.num_blocks, 0x7fffffff) - 1u;

  // ---- gather geometry: wave w, load i covers key rows RPR*(w + 8i) ..
  // +RPR-1 of the tile, all inside one page.  Lane l lands at LDS byte
  // 16*l of that 1 KiB run, i.e. row RPR*(w + 8i) + l/CHUNKS, physical chunk
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
  auto page_ids = [&](int jn, uint32_t (&ids)[NREG]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NREG; ++i) {
      const int page = __builtin_amdgcn_readfirstlane(min(jn * 4 + page_in_tile[i], nblk - 1));
      const uint32_t raw = (uint32_t)bt[page];
      ids[i] = __builtin_amdgcn_readfirstlane(raw > nb_max ? nb_max : raw);
    }
  };
  // element offset of this lane's chunk; positions past the end of the
  // sequence read the last real position instead (finite data whose weight is 0)
  auto src_off = [&](int jn, int i, uint32_t id) __attribute__((always_inline)) -> int64_t {
    const int page = min(jn * 4 + page_in_tile[i], nblk - 1);
    const int last = L - 1 - page * kBlock;
    const int slot = min(keyrow[i] & (kBlock - 1), last);
    return ((((int64_t)id * hkv + g) << 4) + slot) * D + chunk_off[i];
  };
  // bf16 storage: global -> LDS by DMA.  A lane's piece lies at a byte offset
  // within its page run; positions past the end of the sequence take the
  // offset of the last real position instead (lane_bytes, branch-free).  The
  // DMAs themselves (dma) carry no branch either, so the score product can
  // spread them between its matrix instructions instead of every wave
  // issuing all of them at once.
  auto lane_bytes = [&](int jn, uint32_t (&lb)[NREG]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NREG; ++i) {
      const int page = min(jn * 4 + page_in_tile[i], nblk - 1);
      const int last = L - 1 - page * kBlock;
      lb[i] = (uint32_t)((min(keyrow[i] & (kBlock - 1), last) * D + chunk_off[i]) * 2);
    }
  };
  auto dma = [&](uint32_t id, uint32_t lb, int i, const Slot<D>& dst) __attribute__((always_inline)) {
    const int64_t base = (((int64_t)id * hkv + g) << 4) * D;
    const char* ks = reinterpret_cast<const char*>(kpool + base) + lb;
    const char* vs = reinterpret_cast<const char*>(vpool + base) + lb;
    lds_bf16* kd = (lds_bf16*)dst.k.e + lds_off[i];
    lds_bf16* vd = (lds_bf16*)dst.v.e + lds_off[i];
    __builtin_amdgcn_global_load_lds((const void*)ks, (__attribute__((address_space(3))) void*)kd, 16, 0, 0);
    __builtin_amdgcn_global_load_lds((const void*)vs, (__attribute__((address_space(3))) void*)vd, 16, 0, 0);
  };
  // fp32 storage: loads through registers (rounded to bf16), stored once they land
  u32x4 stK[NREG], stV[NREG];
  auto issue_staged = [&](int jn, const uint32_t (&ids)[NREG]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < NREG; ++i) {
      const int64_t off = src_off(jn, i, ids[i]);
      stK[i] = load8(kpool + off);
      stV[i] = load8(vpool + off);
    }
  };
  auto stash = [&](const Slot<D>& dst) __attribute__((always_inline)) {
    if constexpr (!kDirect) {
#pragma unroll
      for (int i = 0; i < NREG; ++i) {
        *reinterpret_cast<u32x4*>(dst.k.e + lds_off[i] + lane * 8) = stK[i];
        *reinterpret_cast<u32x4*>(dst.v.e + lds_off[i] + lane * 8) = stV[i];
      }
    }
  };

  f32x16 o[NB][DT];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[b][dt] = (f32x16){};
  // m_ref: reference max of scale*log2e*score (trails the true max by less
  // than the slack); l_run: this lane's share of sum 2^(s*c - m_ref)
  float m_ref[NB], l_run[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) m_ref[b] = -INFINITY, l_run[b] = 0.f;
  const float c = a.scale_log2;
  const int g16 = (lane >> 4) & 1;
  const int rsel = (lane & 15) >> 2;

  // lane-constant LDS element offsets of the MFMA operand reads; the 32-key
  // half and 16-key group parts are compile-time constants
  int koff[KSTEPS], voff[DT][2];
#pragma unroll
  for (int kk = 0; kk < KSTEPS; ++kk) koff[kk] = l32 * D + (((2 * kk + hh) ^ swz<D>(l32)) << 3);
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int r2 = 0; r2 < 2; ++r2) {
      const int key = 8 * r2 + 4 * hh + rsel;          // key within a 16-key group
      const int dcol = dt * 32 + g16 * 16 + 4 * (lane & 3);
      voff[dt][r2] = key * D + (((dcol >> 3) ^ swz<D>(key)) << 3) + (dcol & 7);
    }
  // ---- S^T = K Q^T of one tile: two independent 32-key accumulator chains
  // per 32-row block, each K fragment read from LDS feeding NB blocks.  With
  // bf16 storage it also issues the gather of the next tile into `fill`
  // (page ids, lane offsets lb), one DMA after each of score steps 1 .. 2*NREG.
  auto qk = [&](const Slot<D>& tl, f32x16 (&s)[NB][2], const uint32_t (&ids)[NREG], const uint32_t (&lb)[NREG],
                const Slot<D>& fill) __attribute__((always_inline)) {
    const __bf16* ks = tl.k.e;
    if constexpr (kDirect) {
#pragma unroll
      for (int i = 0; i < NREG; ++i) dma(ids[i], lb[i], i, fill);
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) s[b][0] = s[b][1] = (f32x16){};
    bf16x8 kf[KSTEPS][2];
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) {
      kf[kk][0] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(ks + koff[kk]));
      kf[kk][1] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(ks + koff[kk] + 32 * D));
    }
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) {
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        s[b][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk][0], qreg[b][kk], s[b][0], 0, 0, 0);
        s[b][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk][1], qreg[b][kk], s[b][1], 0, 0, 0);
      }
    }
    // K fragments read ahead of the products that use them: two steps'
    // worth first, then each pair of products followed by the next pair of
    // reads and (after steps 1 .. 2*NREG) one gather DMA
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int kk = 0; kk < KSTEPS - 2; ++kk) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2 * NB, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      if (kDirect && kk >= 1 && kk <= 2 * NREG) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4 * NB, 0);
  };
  // ---- between tiles: causal mask of tile j (only tiles reaching past the
  // tile's first query), row max, and the reference-max update.  The
  // reference only moves when a tile max passes it by more than the slack;
  // O and l are then rescaled (rare after the first tiles).
  // Element e of half h of a lane's scores is key j*KT + 4*hh + koff(h, e)
  // with koff(h, e) = 32h + 8(e/4) + e%4 in 0..59: the masks compare that
  // constant against one per-lane threshold, so no key index is formed.
  auto settle = [&](int j, f32x16 (&s)[NB][2]) __attribute__((always_inline)) {
    if (j * KT + KT - 1 > lim_min) {
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const int thr = lim[b] - j * KT - 4 * hh;        // keys past lim: koff > thr
#pragma unroll
        for (int half = 0; half < 2; ++half)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (half * 32 + 8 * (e >> 2) + (e & 3) > thr) s[b][half][e] = -INFINITY;
      }
    }
    if (j * KT < kbeg) {   // first tile of a range that starts inside it
      const int thr = kbeg - j * KT - 4 * hh;          // keys before kbeg: koff < thr
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int half = 0; half < 2; ++half)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (half * 32 + 8 * (e >> 2) + (e & 3) < thr) s[b][half][e] = -INFINITY;
    }
    float alpha[NB];
    bool moved = false;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      float mx = -INFINITY;
#pragma unroll
      for (int half = 0; half < 2; ++half)
#pragma unroll
        for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[b][half][e]);
      const float mxc = pair_max(mx) * c;
      const float m_new = (mxc > m_ref[b] + kRescaleSlack) ? mxc : m_ref[b];
      // 1 when unchanged, 0 when leaving -inf; kept at 1 while the row has
      // seen no visible key (a key split can lie wholly past a row's limit)
      alpha[b] = (m_new == -INFINITY) ? 1.0f : __builtin_amdgcn_exp2f(m_ref[b] - m_new);
      m_ref[b] = m_new;
      l_run[b] *= alpha[b];
      moved = moved || alpha[b] != 1.0f;
    }
    if (__builtin_amdgcn_ballot_w64(moved) != 0) {
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[b][dt] *= alpha[b];
    }
  };
  // ---- probabilities of a settled tile: P^T as the B operand of the value
  // product (key group kg = 16 keys); the row sum adds the bf16 values the
  // value product uses
  auto probs = [&](f32x16 (&s)[NB][2], bf16x8 (&pb)[NB][4]) __attribute__((always_inline)) {
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const float m_use = (m_ref[b] == -INFINITY) ? 0.f : m_ref[b];
      float rs = 0.f;
#pragma unroll
      for (int kg = 0; kg < 4; ++kg) {
        const int half = kg >> 1, b0 = (kg & 1) * 8;
        u32x4 wv;
#pragma unroll
        for (int q2 = 0; q2 < 4; ++q2) {
          const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[b][half][b0 + 2 * q2], c, -m_use));
          const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(s[b][half][b0 + 2 * q2 + 1], c, -m_use));
          const bf16x2 pp = __builtin_convertvector((f32x2){p0, p1}, bf16x2);
          rs = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, rs, false);
          wv[q2] = __builtin_bit_cast(unsigned, pp);
        }
        pb[b][kg] = __builtin_bit_cast(bf16x8, wv);
      }
      l_run[b] += rs;
    }
  };
  // ---- O^T += V^T P^T; V^T comes from the row-major tile by transposed
  // reads, each fragment feeding NB MFMAs
  auto pv = [&](const Slot<D>& tl, const bf16x8 (&pb)[NB][4]) __attribute__((always_inline)) {
    const lds_bf16* vl = (const lds_bf16*)tl.v.e;
#pragma unroll
    for (int kg = 0; kg < 4; ++kg) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const bf16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vl + voff[dt][0] + kg * 16 * D));
        const bf16x4 v2 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vl + voff[dt][1] + kg * 16 * D));
        const bf16x8 vf = __builtin_shufflevector(v1, v2, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
        for (int b = 0; b < NB; ++b)
          o[b][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[b][kg], o[b][dt], 0, 0, 0);
      }
    }
  };

  // ---- main loop.  Step t computes tile t (scores, settle, probabilities,
  // value product) and, inside the score product, gathers tile t+1 into the
  // other slot (its page ids were fetched a step earlier; past the last
  // tile the gather still reads clamped, in-bounds pages into a slot no one
  // reads).  The wait + barrier at the end publishes tile t+1 and frees the
  // slot of tile t for the gather of tile t+2.
  const int n = j1 - j0;
  uint32_t ids[NREG], lb[NREG];
  page_ids(j0, ids);
  if (n > 0) {
    if constexpr (kDirect) {
      lane_bytes(j0, lb);
#pragma unroll
      for (int i = 0; i < NREG; ++i) dma(ids[i], lb[i], i, tile0);
    } else {
      issue_staged(j0, ids);
      stash(tile0);
    }
  }
  page_ids(j0 + 1, ids);
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
  __syncthreads();
  f32x16 s_cur[NB][2];
  bf16x8 pb[NB][4];
  auto step = [&](int t, const Slot<D>& cur, const Slot<D>& fill) __attribute__((always_inline)) {
    if constexpr (kDirect) {
      lane_bytes(j0 + t + 1, lb);
    } else if (t + 1 < n) {
      issue_staged(j0 + t + 1, ids);
      stash(fill);
    }
    qk(cur, s_cur, ids, lb, fill);
    page_ids(j0 + t + 2, ids);
    settle(j0 + t, s_cur);
    probs(s_cur, pb);
    pv(cur, pb);
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();
  };
  for (int t = 0; t < n; t += 2) {
    step(t, tile0, tile1);
    if (t + 1 >= n) break;
    step(t + 1, tile1, tile0);
  }

  // ---- epilogue
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const float l_tot = pair_sum(l_run[b]);
    if (!row_valid[b]) continue;
    if (a.direct) {
      const float inv = 1.0f / l_tot;
      T* op = reinterpret_cast<T*>(a.out) + qrow[b] * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int d = dt * 32 + 8 * i + 4 * hh;
          store4(op + d, o[b][dt][4 * i] * inv, o[b][dt][4 * i + 1] * inv, o[b][dt][4 * i + 2] * inv,
                 o[b][dt][4 * i + 3] * inv);
        }
      if (a.lse != nullptr && hh == 0) a.lse[qrow[b]] = (m_ref[b] + __builtin_log2f(l_tot)) * kLn2;
    } else {
      const int64_t prow = (int64_t)(part_base + split) * a.total_rows * a.num_q_heads + qrow[b];
      float* op = a.part_o + prow * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int d = dt * 32 + 8 * i + 4 * hh;
          store4(op + d, o[b][dt][4 * i], o[b][dt][4 * i + 1], o[b][dt][4 * i + 2], o[b][dt][4 * i + 3]);
        }
      if (hh == 0) {
        a.part_ml[prow * 2] = m_ref[b];
        a.part_ml[prow * 2 + 1] = l_tot;
      }
    }
  }
}

// Merge the per-split partial results of each row (fixed split order):
//   m* = max_s m_s,  w_s = 2^(m_s - m*),  out = sum_s w_s O_s / sum_s w_s l_s.
// One thread per 16 columns of a row: four 16-byte loads per split in flight,
// and each split's (m, l) read once per 16 columns.
template <typename T, int D>
__global__ __launch_bounds__(256) void extend_combine_kernel(const CombineArgs a) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // (row, 16-column group)
  constexpr int Q16 = D / 16;
  if (idx >= a.rows * Q16) return;
  const int64_t row = idx / Q16;
  const int c16 = (int)(idx - row * Q16) * 16;
  float mstar = -INFINITY;
  for (int s = 0; s < a.nsplit; ++s) mstar = fmaxf(mstar, a.part_ml[(s * a.rows + row) * 2]);
  float lsum = 0.f;
  f32x4 acc[4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  for (int s = 0; s < a.nsplit; ++s) {
    const int64_t pr = s * a.rows + row;
    const float m = a.part_ml[pr * 2];
    const float w = (m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m - mstar);
    lsum += w * a.part_ml[pr * 2 + 1];
    const f32x4* src = reinterpret_cast<const f32x4*>(a.part_o + pr * D + c16);
    f32x4 v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = src[k];
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[k] += w * v[k];
  }
  const float inv = 1.0f / lsum;
#pragma unroll
  for (int k = 0; k < 4; ++k)
    store4(reinterpret_cast<T*>(a.out) + row * D + c16 + 4 * k, acc[k][0] * inv, acc[k][1] * inv, acc[k][2] * inv,
           acc[k][3] * inv);
  if (a.lse != nullptr && c16 == 0) a.lse[row] = (mstar + __builtin_log2f(lsum)) * kLn2;
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
  const int64_t n = a.rows * (head_dim / 16);
  dim3 g((unsigned)((n + 255) / 256)), b(256);
  if (dtype == 0 && head_dim == 128) hipLaunchKernelGGL((extend_combine_kernel<__bf16, 128>), g, b, 0, stream, a);
  else if (dtype == 0 && head_dim == 64) hipLaunchKernelGGL((extend_combine_kernel<__bf16, 64>), g, b, 0, stream, a);
  else if (dtype == 1 && head_dim == 128) hipLaunchKernelGGL((extend_combine_kernel<float, 128>), g, b, 0, stream, a);
  else hipLaunchKernelGGL((extend_combine_kernel<float, 64>), g, b, 0, stream, a);
  return hipGetLastError();
}

}  // namespace kvt
