// basp_attn_bwd.hip -- backward of the causal GQA attention forward.
//
// For the loss sum(O * dO) the gradients follow from the scaled dot-product
// definition (Sec. II-A of the paper):
//   P_ij  = exp(scale q_i.k_j - LSE_i)           (recomputed from the LSE)
//   D_i   = sum_e dO_i[e] O_i[e]
//   dS_ij = P_ij (dO_i . v_j - D_i)
//   dV_j  = sum_{h in group} sum_{i>=j} P_ij dO_i
//   dK_j  = scale sum_{h in group} sum_{i>=j} dS_ij q_i
//   dQ_i  = scale sum_{j<=i} dS_ij k_j
// Kernels, all deterministic (no atomics):
//   bwd_pre    per (sequence, head, row): LSE in log2 units and -D, in two
//              planes whose rows are padded to a multiple of 64 (zeros)
//   bwd_kv     key-stationary, dV and dK together: a workgroup owns 128 keys
//              of one kv head and sweeps the query rows at or after them (one
//              row chunk of them), for every query head of the GQA group,
//              accumulating in registers
//   bwd_reduce sums the row-chunk partials of dK and dV in chunk order
//   bwd_dq     query-stationary: like the forward, a workgroup owns 256
//              rows of one query head and sweeps the keys up to the diagonal
// gfx950 mapping
//   * v_mfma_f32_32x32x16_bf16 with fp32 accumulation.  The operand order
//     puts every elementwise step (P, dS) in the accumulator layout and feeds
//     it to the next product without a round trip through LDS.  Operands read
//     along the sequence (Q^T, dO^T, K^T) come from the same row-major LDS
//     tiles through ds_read_b64_tr_b16, in the order the accumulator holds P
//     and dS.
//   * the streamed tiles (and, for bwd_kv, the rows' LSE2 and -D) are
//     copied HBM -> LDS by buffer loads that write LDS directly (rows past S
//     arrive as zeros): bwd_dq into a ring of four stages, two tiles ahead;
//     bwd_kv into two stages, one step ahead (measured as fast, and its
//     unmasked loop then runs two steps per iteration, one per stage, so
//     every LDS address is a lane offset plus an immediate).  Each wave
//     waits only for its own copies and passes a fence-free barrier.
//   * both passes run two waves per SIMD (8 waves: bwd_kv 32 keys and one
//     32-row half of each step per wave, bwd_dq 32 rows per wave), which
//     raise their issue priority over the accumulating products so that one
//     wave's elementwise work overlaps the other's MFMAs.
//   * O and the gradients are addressed through row views: the local
//     head-sharded tensors, or (SH) the G sequence shards of the exchange in
//     place (row counts multiples of 256: a workgroup's rows or keys lie in
//     one shard).  Q, K, V and dO, which the passes stream once per tile of
//     the other side, are always local one-buffer views (the in-place entry
//     point packs them first).
#include <math.h>

#include <type_traits>

#include "basp_device.hpp"
#include "basp_internal.hpp"

namespace basp {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kPreThreads = 256;
constexpr int kStages = 4;
// Instruction classes of __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedMfma = 0x008;
constexpr int kSchedDsRead = 0x100;

// Order the LDS operand reads of a run of MFMAs that each take R reads:
// the first A reads up front, then one MFMA per R further reads.
template <int NMFMA, int R, int A>
__device__ __forceinline__ void sched_reads_ahead() {
  __builtin_amdgcn_sched_group_barrier(kSchedDsRead, A, 0);
#pragma unroll
  for (int i = 0; i < NMFMA - A / R; ++i) {
    __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
    __builtin_amdgcn_sched_group_barrier(kSchedDsRead, R, 0);
  }
  __builtin_amdgcn_sched_group_barrier(kSchedMfma, A / R, 0);
}

// ---------------------------------------------------------------- bwd_pre
// One group of D/8 lanes per (beta, row, head) of the padded planes, rows
// r = (beta*Sp + i)*Hl + h; 16-byte loads of O and dO.  Writes
//   lp[beta][h][i] = LSE * log2(e),  np[beta][h][i] = -D_i   (i < S)
// and zeros for the padding rows S <= i < Sp.
template <int D, bool SH>
__global__ __launch_bounds__(kPreThreads) void bwd_pre_kernel(
    const RowView ov, const RowView dov, const float *__restrict__ lse, float *__restrict__ lp,
    float *__restrict__ np, long long rows /* b*Sp*Hl */, int S, int Sp, int Hl) {
  constexpr int LPR = D <= 64 ? 8 : 16;  // lanes per row (a power of two >= D/8)
  const long long gid = (long long)blockIdx.x * kPreThreads + threadIdx.x;
  const long long r = gid / LPR;
  const int sub = (int)(gid % LPR);
  const long long bi = r / Hl;
  const int h = (int)(r - bi * Hl);
  const int beta = (int)(bi / Sp), i = (int)(bi - (long long)beta * Sp);
  float acc = 0.f;
  if (r < rows && i < S && sub < D / 8) {
    const uint16_t *orow, *drow;
    if constexpr (SH) {
      uint32_t left;
      orow = view_row<true, const uint16_t>(ov, beta, i, h, D, left);
      drow = view_row<false, const uint16_t>(dov, beta, i, h, D, left);
    } else {  // local [b][S][Hl][D]
      const size_t e = (((size_t)beta * S + i) * Hl + h) * D;
      orow = static_cast<const uint16_t *>(ov.p[0]) + e;
      drow = static_cast<const uint16_t *>(dov.p[0]) + e;
    }
    const u32x4 a = reinterpret_cast<const u32x4 *>(orow)[sub];
    const u32x4 b = reinterpret_cast<const u32x4 *>(drow)[sub];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc += bf16_bits_to_f32(a[i] & 0xFFFFu) * bf16_bits_to_f32(b[i] & 0xFFFFu);
      acc += bf16_bits_to_f32(a[i] >> 16) * bf16_bits_to_f32(b[i] >> 16);
    }
  }
#pragma unroll
  for (int off = LPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
  if (r < rows && sub == 0) {
    const size_t row = (size_t)beta * Hl + h;
    lp[row * Sp + i] = i < S ? lse[row * S + i] * kLog2e : 0.f;
    np[row * Sp + i] = i < S ? -acc : 0.f;
  }
}

// ------------------------------------------------------ bwd_kv (dV and dK)
// Key-stationary, dV and dK in one pass.  A workgroup of 8 waves, two per
// SIMD, owns 128 keys of one kv head and sweeps 64-row query steps for all
// query heads of the GQA group.  Wave w takes keys 32 (w % 4) .. +31 and the
// 32-row half w / 4 of every step, and forms
//   S^T = K Q^T and dP^T = V dO^T       (K of its keys in registers; V too
//                                        below d = 128, else from LDS)
//   P = exp2(S c - LSE2),  dS = P (dP - D)
//   dV^T += dO^T P  and  dK^T += Q^T dS  (accumulated in registers)
// so S is formed once for both gradients.  The two waves of a key block
// (w, w + 4, which share a SIMD) hold partial sums over their halves and add
// them once per unit, through LDS, in that order.  Each wave raises its issue
// priority over its accumulating products, so that the two waves of a SIMD
// drift apart and one's elementwise work overlaps the other's MFMAs.
constexpr int kKvWaves = 8;
constexpr int kKvThreads = 64 * kKvWaves;
constexpr int kKN = 128;  // keys per workgroup (32 per key block)
static_assert(kKN == kKvKeys, "work units assume 128 keys per workgroup");
constexpr int kQM = 64;   // query rows per step (two 32-row halves)

template <int D>
struct KvCfg {
  static constexpr int DC = HeadDim<D>::DC;
  static constexpr int LW = HeadDim<D>::LW;
  static constexpr int TILE_BYTES = kQM * LW * 2;   // a step's Q or dO rows
  static constexpr int KT_BYTES = kKN * LW * 2;     // the workgroup's V rows
  static constexpr int AUX_BYTES = 1024;            // LSE2, then -D, of the step's rows
  static constexpr int NS = DC / 16;
  static constexpr int NE = DC / 32;
  static constexpr int CPR = LW / 8;
  static constexpr int DMA_PER_WAVE = kQM * CPR / kKvThreads;     // 1 KB copies per tile
  static constexpr int KV_DMA_PER_WAVE = kKN * CPR / kKvThreads;  // for the V tile
  static constexpr bool V_REGS = D < 128;  // V of the wave's keys fits in registers
};

template <int D, bool SH>
__global__ __launch_bounds__(kKvThreads, 1) void bwd_kv_kernel(
    const RowView qv, const RowView kv, const RowView vv, const RowView dov,
    const float *__restrict__ lp, uint32_t plane_bytes /* np - lp */, const RowView dvv,
    const RowView dkv, size_t chunk_elems, int S, int Sp, int Hl, int Hkl, int n_rep,
    int kvheads_total, int ktiles, int nchunks, int chunk_tiles, float c /* scale*log2e */,
    float dk_scale) {
  using C = KvCfg<D>;
  using T = LdsTile<C::LW>;
  // LDS: Q tiles of the two ring stages, their dO tiles, their (LSE2, -D)
  // blocks, then (d = 128) the V tile of the workgroup's keys.  After the
  // last step the same bytes hold the second waves' partial sums: 1 KB per
  // (key block, tensor, register group).
  constexpr int kDoRegion = 2 * C::TILE_BYTES;
  constexpr int kAuxRegion = 4 * C::TILE_BYTES;
  constexpr int kKvRegion = kAuxRegion + 2 * C::AUX_BYTES;
  constexpr int kPartBytes = kKvWaves / 2 * 2 * C::NE * 4 * 1024;
  constexpr int kRingBytes = kKvRegion + (C::V_REGS ? 0 : C::KT_BYTES);
  constexpr int kLdsBytes = kRingBytes > kPartBytes ? kRingBytes : kPartBytes;
  __shared__ __attribute__((aligned(16))) unsigned char smem[kLdsBytes];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kw = w & 3, h = w >> 2;  // key block, row half
  const int l32 = lane & 31, hh = lane >> 5;
  const int L = blockIdx.x;
  const int hb = L % kvheads_total;
  int kt, ch;
  kv_unit(L / kvheads_total, nchunks, chunk_tiles, kt, ch);
  if (kt >= ktiles) return;  // workgroup-uniform
  const int beta = hb / Hkl, kvh = hb % Hkl;
  const int k0 = kt * kKN;
  const int chunk_rows = chunk_tiles * kKvKeys;
  const int r_lo = max(k0, ch * chunk_rows), r_hi = min(S, (ch + 1) * chunk_rows);
  if (r_lo >= r_hi) return;
  const int wk0 = k0 + 32 * kw;
  const int key = wk0 + l32;

  const uint32_t q_row_bytes = qv.row_elems * 2, kv_row_bytes = kv.row_elems * 2;
  const uint32_t smem_lds = lds_addr_of(smem);
  // K of this lane's key as B operands in registers; V too below d = 128,
  // where it fits, else the V tile of the workgroup's keys in LDS (rows past
  // S arrive as zeros).
  constexpr bool kVRegs = C::V_REGS;
  bf16x8 kf[C::NS], vf[kVRegs ? C::NS : 1];
  {
    uint32_t left;
    const rsrc_t rk = make_rsrc(view_row<false, const uint16_t>(kv, beta, k0, kvh, D, left),
                                left * kv_row_bytes);
#pragma unroll
    for (int s = 0; s < C::NS; ++s) {
      const uint32_t off = (uint32_t)(key - k0) * kv_row_bytes + (2 * s + hh) * 16;
      kf[s] = 2 * s < D / 8 ? as_bf16x8(buf_load16(rk, off)) : bf16x8{};  // columns past D
    }
    if constexpr (kVRegs) {
      const rsrc_t rv = make_rsrc(view_row<false, const uint16_t>(vv, beta, k0, kvh, D, left),
                                  left * kv_row_bytes);
#pragma unroll
      for (int s = 0; s < C::NS; ++s) {
        const uint32_t off = (uint32_t)(key - k0) * kv_row_bytes + (2 * s + hh) * 16;
        vf[s] = 2 * s < D / 8 ? as_bf16x8(buf_load16(rv, off)) : bf16x8{};
      }
    }
    wait_vmcnt<0>();  // retire the tracked loads before untracked copies start
    if constexpr (!kVRegs) {
      const u32x4 rv = make_rsrc_words(
          view_row<false, const uint16_t>(vv, beta, k0, kvh, D, left), left * kv_row_bytes);
#pragma unroll
      for (int i = 0; i < C::KV_DMA_PER_WAVE; ++i) {
        const int pos = (w * C::KV_DMA_PER_WAVE + i) * 64 + lane;
        const uint32_t off = dma_src_off<C::LW, D>(pos, kv_row_bytes);
        buf_load16_lds_async(rv, off,
                             smem_lds + kKvRegion + (w * C::KV_DMA_PER_WAVE + i) * 1024);
      }
    }
  }

  f32x16 accv[C::NE], acck[C::NE];
#pragma unroll
  for (int n = 0; n < C::NE; ++n)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      accv[n][r] = 0.f;
      acck[n][r] = 0.f;
    }

  const int steps_per_head = (r_hi - r_lo + kQM - 1) / kQM;
  const int nsteps = steps_per_head * n_rep;

  uint32_t g_off[C::DMA_PER_WAVE];
#pragma unroll
  for (int i = 0; i < C::DMA_PER_WAVE; ++i)
    g_off[i] = dma_src_off<C::LW, D>((w * C::DMA_PER_WAVE + i) * 64 + lane, q_row_bytes);
  // A of S^T (Q) and dP^T (dO): row 32h + l32 of the step, chunk 2s + hh.
  // B of dP^T from LDS (V, at d = 128): row 32kw + l32 of the V tile, same
  // chunk.
  int a_off[C::NS], b_off[kVRegs ? 1 : C::NS];
#pragma unroll
  for (int s = 0; s < C::NS; ++s) {
    a_off[s] = T::off(32 * h + l32, 2 * s + hh);
    asm volatile("" : "+v"(a_off[s]));
    if constexpr (!kVRegs) {
      b_off[s] = kKvRegion + T::off(32 * kw + l32, 2 * s + hh);
      asm volatile("" : "+v"(b_off[s]));
    }
  }
  // Transposed A of dV^T / dK^T: rows 32h + 16*s2 + 4hh (+8), columns 32n + 16*((lane/16)&1).
  int t_off[C::NE][2];
#pragma unroll
  for (int n = 0; n < C::NE; ++n)
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      t_off[n][x] =
          tr_piece_off<C::LW>(32 * h + 4 * hh + 8 * x, 32 * n + 16 * ((lane >> 4) & 1), lane);
      asm volatile("" : "+v"(t_off[n][x]));
    }
  // This lane's first (LSE2, -D) value of its half in a stage's aux block.
  int aux_lane = kAuxRegion + 4 * 32 * h + 16 * hh;
  asm volatile("" : "+v"(aux_lane));
  auto launder_offsets = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int s = 0; s < C::NS; ++s) {
      asm volatile("" : "+v"(a_off[s]));
      if constexpr (!kVRegs) asm volatile("" : "+v"(b_off[s]));
    }
#pragma unroll
    for (int n = 0; n < C::NE; ++n) {
      asm volatile("" : "+v"(t_off[n][0]));
      asm volatile("" : "+v"(t_off[n][1]));
    }
    asm volatile("" : "+v"(aux_lane));
  };

  const int nmask_ph = kv_masked_steps(k0, r_lo, steps_per_head, kQM);
  // Copy state.  Steps are copied strictly in order, one ahead of use: the
  // next one to copy is step ld_t of head ld_hr of the group, first row
  // ld_i0, and rq, rd, ra are its resources (Q and dO rows from ld_i0 on,
  // the head's (LSE2, -D) planes).  They advance by one step's rows at a
  // time and are rebuilt per head, so a step costs a few scalar additions.
  int ld_hr = 0, ld_t = 0, ld_i0 = r_lo;
  u32x4 rq, rd, ra;
  // Lanes 0-15 copy the step's 64 LSE2 values, lanes 16-31 its 64 -D values
  // (the padded planes hold every row the steps reach); the other lanes
  // read zeros.
  const uint32_t aux_lane_off = lane < 16   ? 16u * lane
                                : lane < 32 ? plane_bytes + 16u * (lane - 16)
                                            : kZeroOffset;
  auto head_resources = [&]() __attribute__((always_inline)) {
    const int hq = kvh * n_rep + ld_hr;
    uint32_t left;  // rows from r_lo to the sequence's end; rows past it read as zeros
    rq = make_rsrc_words(view_row<false, const uint16_t>(qv, beta, r_lo, hq, D, left),
                         left * q_row_bytes);
    rd = make_rsrc_words(view_row<false, const uint16_t>(dov, beta, r_lo, hq, D, left),
                         left * q_row_bytes);
    ra = make_rsrc_words(lp + ((size_t)beta * Hl + hq) * Sp, plane_bytes + (uint32_t)Sp * 4);
  };
  auto advance = [&](u32x4 &r, uint32_t bytes) __attribute__((always_inline)) {
    const uint64_t a = (((uint64_t)r[1] << 32) | r[0]) + bytes;  // 48-bit base, stride 0
    r[0] = (uint32_t)a;
    r[1] = (uint32_t)(a >> 32);
    r[2] -= bytes;  // rows left from the new first row (at least one)
  };
  head_resources();
  // Copies of step st into ring stage st % 2: Q and dO rows (every wave its
  // share), the rows' LSE2 and -D (wave 0, 1 KB of which 512 B are used).
  auto load_step = [&](int st) __attribute__((always_inline)) {
    const uint32_t sq = (uint32_t)st & 1;
    const uint32_t stage = smem_lds + sq * C::TILE_BYTES;
#pragma unroll
    for (int i = 0; i < C::DMA_PER_WAVE; ++i) {
      const uint32_t lds = stage + (w * C::DMA_PER_WAVE + i) * 1024;
      buf_load16_lds_async(rq, g_off[i], lds);
      buf_load16_lds_async(rd, g_off[i], lds + kDoRegion);
    }
    if (w == 0)
      buf_load16_lds_async(ra, aux_lane_off + (uint32_t)ld_i0 * 4,
                           smem_lds + kAuxRegion + sq * C::AUX_BYTES);
    if (++ld_t == steps_per_head) {
      ld_t = 0;
      ld_i0 = r_lo;
      if (++ld_hr < n_rep) head_resources();
    } else {
      ld_i0 += kQM;
      advance(rq, kQM * q_row_bytes);
      advance(rd, kQM * q_row_bytes);
    }
  };
  // 16 values (rows 32h + 8g + 4hh + {0..3} of the step) of part `part`
  // (0: LSE2, 1: -D) of stage stg's aux block.
  auto aux_rows = [&](int stg, int part) __attribute__((always_inline)) {
    const unsigned char *a = smem + aux_lane + stg * C::AUX_BYTES + 256 * part;
    f32x16 v;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 x = *reinterpret_cast<const f32x4 *>(a + 4 * 8 * g);
#pragma unroll
      for (int y = 0; y < 4; ++y) v[4 * g + y] = x[y];
    }
    return v;
  };
  // One step's half for this wave.  lim: rows of the half whose offset is
  // below lim precede the key (masked); 0 or less for none.
  auto step = [&](int stg, int lim, auto mask_tag) __attribute__((always_inline)) {
    constexpr bool MASK = decltype(mask_tag)::value;
    const unsigned char *Qs = smem + stg * C::TILE_BYTES, *dOs = Qs + kDoRegion;
    f32x16 sacc, pacc;
    {
      const f32x16 negd = aux_rows(stg, 1);
#pragma unroll
      for (int s = 0; s < C::NS; ++s) {
        const bf16x8 aq = *reinterpret_cast<const bf16x8 *>(Qs + a_off[s]);
        const bf16x8 ad = *reinterpret_cast<const bf16x8 *>(dOs + a_off[s]);
        bf16x8 bv;
        if constexpr (kVRegs) bv = vf[s];
        else bv = *reinterpret_cast<const bf16x8 *>(smem + b_off[s]);
        sacc = mfma32x32x16(aq, kf[s], s == 0 ? f32x16{} : sacc);
        pacc = mfma32x32x16(ad, bv, s == 0 ? negd : pacc);
      }
    }
    bf16x8 bp[2], bds[2];
    {
      const f32x16 lse2 = aux_rows(stg, 0);
      float ds[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float p = fast_exp2(fmaf(sacc[r], c, -lse2[r]));
        if (MASK && 8 * (r >> 2) + (r & 3) < lim) p = 0.f;
        sacc[r] = p;
        ds[r] = p * pacc[r];
      }
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const int b8 = 8 * s2;
        bp[s2] = as_bf16x8(u32x4{pack_bf16x2(sacc[b8 + 0], sacc[b8 + 1]),
                                 pack_bf16x2(sacc[b8 + 2], sacc[b8 + 3]),
                                 pack_bf16x2(sacc[b8 + 4], sacc[b8 + 5]),
                                 pack_bf16x2(sacc[b8 + 6], sacc[b8 + 7])});
        bds[s2] = as_bf16x8(u32x4{pack_bf16x2(ds[b8 + 0], ds[b8 + 1]),
                                  pack_bf16x2(ds[b8 + 2], ds[b8 + 3]),
                                  pack_bf16x2(ds[b8 + 4], ds[b8 + 5]),
                                  pack_bf16x2(ds[b8 + 6], ds[b8 + 7])});
      }
    }
    wave_priority<1>();
#pragma unroll
    for (int n = 0; n < C::NE; ++n)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const int ro = s2 * 16 * T::ROW_BYTES;
        const bf16x8 av = tr_operand(dOs, t_off[n][0] + ro, t_off[n][1] + ro);
        accv[n] = mfma32x32x16(av, bp[s2], accv[n]);
        const bf16x8 ak = tr_operand(Qs, t_off[n][0] + ro, t_off[n][1] + ro);
        acck[n] = mfma32x32x16(ak, bds[s2], acck[n]);
      }
    sched_reads_ahead<4 * C::NE, 2, 4>();
    __builtin_amdgcn_sched_barrier(0);
    wave_priority<0>();
  };

  load_step(0);
  // Two stages: step st's copies (and, before step 0, the K/V tiles)
  // landed, then the barrier, after which stage (st+1) % 2 is free.
  auto begin_step = [&](int st) __attribute__((always_inline)) {
    wait_vmcnt<0>();
    barrier_no_fence();
    if (st + 1 < nsteps) load_step(st + 1);
  };
  int st = 0;
  for (int hr = 0; hr < n_rep; ++hr) {
    for (int t = 0; t < nmask_ph; ++t, ++st) {
      begin_step(st);
      const int i0 = r_lo + t * kQM;
      if (i0 + 32 * h + 31 >= wk0)  // wave-uniform: some row of the half reaches a key
        step(st & 1, key - i0 - 32 * h - 4 * hh, std::true_type{});
    }
    int t = nmask_ph;
    if ((st & 1) && t < steps_per_head) {
      begin_step(st);
      step(1, 0, std::false_type{});
      ++t;
      ++st;
    }
    for (; t + 1 < steps_per_head; t += 2, st += 2) {
      launder_offsets();
      begin_step(st);
      step(0, 0, std::false_type{});
      begin_step(st + 1);
      step(1, 0, std::false_type{});
    }
    if (t < steps_per_head) {
      begin_step(st);
      step(0, 0, std::false_type{});
      ++st;
    }
  }

  // The pair's partial sums: the second waves put theirs in LDS (every step
  // is done: no copy in flight, nothing left to read), the first add them.
  barrier_no_fence();
  // Slot of (key block, tensor, register group n*4 + g): 1 KB, lane l's 16
  // bytes at 16 l.
  auto slot = [&](int tensor, int n, int g) __attribute__((always_inline)) {
    return smem + (((kw * 2 + tensor) * C::NE + n) * 4 + g) * 1024 + 16 * lane;
  };
  if (h == 1) {
#pragma unroll
    for (int n = 0; n < C::NE; ++n)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        *reinterpret_cast<f32x4 *>(slot(0, n, g)) =
            f32x4{accv[n][4 * g], accv[n][4 * g + 1], accv[n][4 * g + 2], accv[n][4 * g + 3]};
        *reinterpret_cast<f32x4 *>(slot(1, n, g)) =
            f32x4{acck[n][4 * g], acck[n][4 * g + 1], acck[n][4 * g + 2], acck[n][4 * g + 3]};
      }
  }
  __syncthreads();
  if (h == 1 || key >= S) return;
  uint32_t left;
  float *ov = view_row<true, float>(dvv, beta, k0, kvh, D, left) + (size_t)ch * chunk_elems +
              (size_t)(key - k0) * dvv.row_elems;
  float *ok = view_row<true, float>(dkv, beta, k0, kvh, D, left) + (size_t)ch * chunk_elems +
              (size_t)(key - k0) * dkv.row_elems;
#pragma unroll
  for (int n = 0; n < C::NE; ++n)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      if (32 * n + 8 * g >= D) continue;  // padding columns
      const f32x4 pv = *reinterpret_cast<const f32x4 *>(slot(0, n, g));
      const f32x4 pk = *reinterpret_cast<const f32x4 *>(slot(1, n, g));
      *reinterpret_cast<f32x4 *>(ov + 32 * n + 8 * g + 4 * hh) =
          f32x4{accv[n][4 * g] + pv[0], accv[n][4 * g + 1] + pv[1], accv[n][4 * g + 2] + pv[2],
                accv[n][4 * g + 3] + pv[3]};
      *reinterpret_cast<f32x4 *>(ok + 32 * n + 8 * g + 4 * hh) =
          f32x4{(acck[n][4 * g] + pk[0]) * dk_scale, (acck[n][4 * g + 1] + pk[1]) * dk_scale,
                (acck[n][4 * g + 2] + pk[2]) * dk_scale, (acck[n][4 * g + 3] + pk[3]) * dk_scale};
    }
}

// ---------------------------------------------------------------- bwd_reduce
// dK or dV of a key = the sum of the partial sums of the row chunks that
// exist for its key tile, added in chunk order (deterministic).  One thread
// per 4 consecutive elements of a key's row of the rank's kv heads; grid.y is
// the sequence.  The partials are local [chunk][b][S][Hkl][d]; the result
// goes through the output view (the rank's heads are contiguous in a row).
__global__ __launch_bounds__(kPreThreads) void bwd_reduce_kernel(
    const float *__restrict__ part, const RowView outv, uint32_t row_quads /* Hkl*D/4 */,
    FastDiv by_row_quads, uint32_t seq_quads /* S*row_quads */, size_t slice /* b*S*Hkl*D */,
    int d, int nchunks, int chunk_tiles) {
  const uint32_t i = blockIdx.x * kPreThreads + threadIdx.x;
  if (i >= seq_quads) return;
  const int beta = blockIdx.y;
  const uint32_t key = by_row_quads.div(i), cq = i - key * row_quads;
  const size_t e = ((size_t)beta * seq_quads + i) * 4;
  const int first = (int)(key / kKN) / chunk_tiles;  // first chunk the key tile wrote
  f32x4 acc = *reinterpret_cast<const f32x4 *>(part + (size_t)first * slice + e);
  for (int ch = first + 1; ch < nchunks; ++ch) {
    const f32x4 x = *reinterpret_cast<const f32x4 *>(part + (size_t)ch * slice + e);
    acc[0] += x[0];
    acc[1] += x[1];
    acc[2] += x[2];
    acc[3] += x[3];
  }
  uint32_t left;
  *reinterpret_cast<f32x4 *>(view_row<true, float>(outv, beta, key, 0, d, left) + 4 * cq) = acc;
}

// ---------------------------------------------------------------- bwd_dq
constexpr int kDqWaves = 8;
constexpr int kDqThreads = 64 * kDqWaves;
constexpr int kDQM = 32 * kDqWaves;  // query rows per workgroup (32 per wave)
constexpr int kDQN = 64;             // keys per tile

template <int D>
struct DqCfg {
  static constexpr int DC = HeadDim<D>::DC;
  static constexpr int LW = HeadDim<D>::LW;
  static constexpr int TILE_BYTES = kDQN * LW * 2;
  static constexpr int STAGE_BYTES = 2 * TILE_BYTES;  // K, V
  static constexpr int NS = DC / 16;
  static constexpr int NE = DC / 32;
  static constexpr int CPR = LW / 8;
  static constexpr int DMA_PER_WAVE = kDQN * CPR / kDqThreads;
};

template <int D, bool SH>
__global__ __launch_bounds__(kDqThreads, 1) void bwd_dq_kernel(
    const RowView qv, const RowView kv, const RowView vv, const RowView dov,
    const float *__restrict__ lp, const float *__restrict__ np, const RowView dqv, int S, int Sp,
    int Hl, int n_rep, int heads_total, int qtiles, float c, float scale) {
  using C = DqCfg<D>;
  using T = LdsTile<C::LW>;
  // LDS: the K tiles of the kStages ring stages, then their V tiles; with
  // the tile loop unrolled over the stages every operand address is a lane's
  // fixed offset plus an instruction immediate.
  __shared__ __attribute__((aligned(16))) unsigned char smem[kStages * C::STAGE_BYTES];
  constexpr int kVRegion = kStages * C::TILE_BYTES;

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hh = lane >> 5;
  const int L = blockIdx.x;
  const int qt = qtiles - 1 - L / heads_total;
  const int hb = L % heads_total;
  const int beta = hb / Hl, h = hb % Hl, kvh = h / n_rep;
  const int q0 = qt * kDQM;
  const int wrow0 = q0 + 32 * w;
  const int row = wrow0 + l32;

  const uint32_t q_row_bytes = qv.row_elems * 2, kv_row_bytes = kv.row_elems * 2;
  uint32_t left;
  const rsrc_t rq =
      make_rsrc(view_row<false, const uint16_t>(qv, beta, q0, h, D, left), left * q_row_bytes);
  const rsrc_t rd =
      make_rsrc(view_row<false, const uint16_t>(dov, beta, q0, h, D, left), left * q_row_bytes);
  // K and V are local (the in-place entry point packs them): one resource
  // per head for every tile.
  const u32x4 rk = make_rsrc_words(view_row<false, const uint16_t>(kv, beta, 0, kvh, D, left),
                                   left * kv_row_bytes);
  const u32x4 rv = make_rsrc_words(view_row<false, const uint16_t>(vv, beta, 0, kvh, D, left),
                                   left * kv_row_bytes);
  const uint32_t smem_lds = lds_addr_of(smem);

  bf16x8 qf[C::NS], df[C::NS];
#pragma unroll
  for (int s = 0; s < C::NS; ++s) {
    if (2 * s < D / 8) {
      qf[s] = as_bf16x8(buf_load16(rq, (uint32_t)(row - q0) * q_row_bytes + (2 * s + hh) * 16));
      df[s] = as_bf16x8(buf_load16(rd, (uint32_t)(row - q0) * q_row_bytes + (2 * s + hh) * 16));
    } else {  // columns past D
      qf[s] = bf16x8{};
      df[s] = bf16x8{};
    }
  }
  float lse2 = INFINITY, nd = 0.f;  // rows past S: P = 0
  if (row < S) {
    lse2 = lp[((size_t)beta * Hl + h) * Sp + row];
    nd = np[((size_t)beta * Hl + h) * Sp + row];
  }
  // dP^T starts from -D (the accumulator's initial value), so dS = P dP'.
  // (At d = 64 the 16 registers this takes leave room for one workgroup per
  // CU instead of two; measured faster all the same.)
  f32x16 negd;
#pragma unroll
  for (int r = 0; r < 16; ++r) negd[r] = nd;
  wait_vmcnt<0>();  // retire the tracked loads before untracked copies start

  const int kv_end = min(S, q0 + kDQM);
  const int nt = (kv_end + kDQN - 1) / kDQN;

  uint32_t g_off[C::DMA_PER_WAVE];
#pragma unroll
  for (int i = 0; i < C::DMA_PER_WAVE; ++i)
    g_off[i] = dma_src_off<C::LW, D>((w * C::DMA_PER_WAVE + i) * 64 + lane, kv_row_bytes);
  auto load_tile = [&](int t) __attribute__((always_inline)) {
    const uint32_t ks = smem_lds + (t % kStages) * C::TILE_BYTES;
    const uint32_t base = (uint32_t)(t * kDQN) * kv_row_bytes;
#pragma unroll
    for (int i = 0; i < C::DMA_PER_WAVE; ++i) {
      const uint32_t lds = ks + (w * C::DMA_PER_WAVE + i) * 1024;
      buf_load16_lds_async(rk, base + g_off[i], lds);
      buf_load16_lds_async(rv, base + g_off[i], lds + kVRegion);
    }
  };
  // Row l32 (+32 for m = 1), chunk 2s + hh, of the K tile (a_off) and the V
  // tile (v_off).  With 64-wide rows the V region starts within reach of the
  // instruction immediate, so V takes the K offsets.
  constexpr bool kVImm = kVRegion + kStages * C::TILE_BYTES <= 65536;
  int a_off[C::NS], v_off[C::NS];
#pragma unroll
  for (int s = 0; s < C::NS; ++s) {
    a_off[s] = T::off(l32, 2 * s + hh);
    asm volatile("" : "+v"(a_off[s]));
    if constexpr (!kVImm) {
      v_off[s] = a_off[s] + kVRegion;
      asm volatile("" : "+v"(v_off[s]));
    }
  }
  auto v_at = [&](int s) __attribute__((always_inline)) {
    if constexpr (kVImm) return a_off[s] + kVRegion;
    else return v_off[s];
  };
  // Transposed A operand: rows 16*s2 + 4hh (+8), columns 32n + 16*((lane/16)&1).
  int t_off[C::NE][2];
#pragma unroll
  for (int n = 0; n < C::NE; ++n)
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      t_off[n][x] = tr_piece_off<C::LW>(4 * hh + 8 * x, 32 * n + 16 * ((lane >> 4) & 1), lane);
      asm volatile("" : "+v"(t_off[n][x]));
    }

  f32x16 qacc[C::NE];
#pragma unroll
  for (int n = 0; n < C::NE; ++n)
#pragma unroll
    for (int r = 0; r < 16; ++r) qacc[n][r] = 0.f;

  // One 64-key tile in two 32-key halves (keeps the score state at 2 x 16
  // registers).  S^T = K Q^T and dP^T = V dO^T: M = 32 keys, N = this wave's
  // rows; sacc[r] holds key j0 + 32m + 8(r/4) + 4hh + r%4, query row `row`.
  // `st` = t % kStages (a constant in the unrolled loop).
  auto tile = [&](int t, int st, auto mask_tag) __attribute__((always_inline)) {
    constexpr bool MASK = decltype(mask_tag)::value;
    const int j0 = t * kDQN;
    const unsigned char *Ks = smem + st * C::TILE_BYTES;
    const unsigned char *Vs = Ks;  // v_at adds the V region's base
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      if (MASK && j0 + 32 * m > wrow0 + 31) continue;  // wave-uniform: half entirely masked
      f32x16 sacc, pacc;
      {
        const bf16x8 ak = *reinterpret_cast<const bf16x8 *>(Ks + a_off[0] + m * 32 * T::ROW_BYTES);
        const bf16x8 av = *reinterpret_cast<const bf16x8 *>(Vs + v_at(0) + m * 32 * T::ROW_BYTES);
        sacc = mfma32x32x16(ak, qf[0], f32x16{});
        pacc = mfma32x32x16(av, df[0], negd);
      }
#pragma unroll
      for (int s = 1; s < C::NS; ++s) {
        const bf16x8 ak = *reinterpret_cast<const bf16x8 *>(Ks + a_off[s] + m * 32 * T::ROW_BYTES);
        const bf16x8 av = *reinterpret_cast<const bf16x8 *>(Vs + v_at(s) + m * 32 * T::ROW_BYTES);
        sacc = mfma32x32x16(ak, qf[s], sacc);
        pacc = mfma32x32x16(av, df[s], pacc);
      }
      sched_reads_ahead<2 * C::NS, 1, 4>();
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float p = fast_exp2(fmaf(sacc[r], c, -lse2));
        if constexpr (MASK) {
          const int j = j0 + 32 * m + 8 * (r >> 2) + 4 * hh + (r & 3);
          if (j > row) p = 0.f;
        }
        pacc[r] = p * pacc[r];
      }
      bf16x8 sb[2];
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const int b8 = 8 * s2;
        u32x4 ts = {pack_bf16x2(pacc[b8 + 0], pacc[b8 + 1]), pack_bf16x2(pacc[b8 + 2], pacc[b8 + 3]),
                    pack_bf16x2(pacc[b8 + 4], pacc[b8 + 5]), pack_bf16x2(pacc[b8 + 6], pacc[b8 + 7])};
        sb[s2] = as_bf16x8(ts);
      }
      // dQ^T += K^T dS^T: M = head dim, N = rows, K = keys; K^T straight
      // from the row-major K tile, at raised issue priority (see the header).
      wave_priority<1>();
#pragma unroll
      for (int n = 0; n < C::NE; ++n)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const int ro = (2 * m + s2) * 16 * T::ROW_BYTES;
          const bf16x8 a = tr_operand(Ks, t_off[n][0] + ro, t_off[n][1] + ro);
          qacc[n] = mfma32x32x16(a, sb[s2], qacc[n]);
        }
      sched_reads_ahead<2 * C::NE, 2, 4>();
      __builtin_amdgcn_sched_barrier(0);  // keep the two halves apart (register pressure)
      wave_priority<0>();
    }
  };
  auto step = [&](int t) __attribute__((always_inline)) {
    // Stage (t+2) % 4 last held tile t-2, finished by every wave before the
    // barrier of iteration t-1.  With two tiles in flight the wait keeps
    // them; the last two tiles wait for every copy.
    if (t + 2 < nt) {
      load_tile(t + 2);
      wait_vmcnt<4 * C::DMA_PER_WAVE>();
    } else {
      wait_vmcnt<0>();
    }
    barrier_no_fence();
  };
  for (int t = 0; t < 2 && t < nt; ++t) load_tile(t);
  const int t_mask = min(nt, q0 / kDQN);  // tiles before t_mask need no mask
  static_assert(kStages == 4, "the unrolled loop assumes four ring stages");
  int t = 0;
  for (; t + 4 <= t_mask; t += 4) {  // t % 4 == 0
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      step(t + u);
      tile(t + u, u, std::false_type{});
    }
  }
  for (; t < t_mask; ++t) {
    step(t);
    tile(t, t % kStages, std::false_type{});
  }
  for (; t < nt; ++t) {
    step(t);
    if (t * kDQN <= wrow0 + 31) tile(t, t % kStages, std::true_type{});  // wave-uniform
  }

  if (row < S) {
    float *dqr = view_row<SH, float>(dqv, beta, q0, h, D, left) + (size_t)(row - q0) * dqv.row_elems;
#pragma unroll
    for (int n = 0; n < C::NE; ++n)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        if (32 * n + 8 * g >= D) continue;  // padding columns
        f32x4 a = {qacc[n][4 * g] * scale, qacc[n][4 * g + 1] * scale,
                   qacc[n][4 * g + 2] * scale, qacc[n][4 * g + 3] * scale};
        *reinterpret_cast<f32x4 *>(dqr + 32 * n + 8 * g + 4 * hh) = a;
      }
  }
}

template <int D, bool SH>
hipError_t launch_bwd_d(const RowView &q, const RowView &k, const RowView &v, const RowView &o,
                        const float *lse, const RowView &d_o, const RowView &dq,
                        const RowView &dk, const RowView &dv, float *ws, const AttnShape &s,
                        hipStream_t stream) {
  // LSE2 and -D planes, rows padded to a multiple of 64 (every row a
  // key-stationary step reaches).
  const int Sp = bwd_plane_rows(s.S);
  float *lp = ws, *np = ws + (size_t)s.b * s.Hl * Sp;
  const uint32_t plane_bytes = (uint32_t)((size_t)s.b * s.Hl * Sp * 4);
  const float c = s.scale * kLog2e;
  const int n_rep = s.Hl / s.Hkl;

  const long long rows = (long long)s.b * Sp * s.Hl;
  const long long pre_threads = rows * (D <= 64 ? 8 : 16);
  const long long pre_blocks = (pre_threads + kPreThreads - 1) / kPreThreads;
  hipLaunchKernelGGL((bwd_pre_kernel<D, SH>), dim3((unsigned)pre_blocks), dim3(kPreThreads), 0,
                     stream, o, d_o, lse, lp, np, rows, s.S, Sp, s.Hl);

  const int ktiles = (s.S + kKN - 1) / kKN;
  const int kvheads_total = s.b * s.Hkl;
  const BwdChunks ck = bwd_chunks(s);
  const dim3 kv_grid((unsigned)(ck.units * kvheads_total));
  RowView dv_out = dv, dk_out = dk;
  size_t chunk_elems = 0;
  float *dv_part = nullptr, *dk_part = nullptr;
  if (ck.n > 1) {  // partial sums in the workspace, reduced below
    chunk_elems = (size_t)kvheads_total * s.S * D;
    dv_part = ws + ck.part_offset_floats;
    dk_part = dv_part + (size_t)ck.n * chunk_elems;
    dv_out = local_view(dv_part, s.S, s.Hkl, D);
    dk_out = local_view(dk_part, s.S, s.Hkl, D);
  }
  hipLaunchKernelGGL((bwd_kv_kernel<D, SH>), kv_grid, dim3(kKvThreads), 0, stream, q, k, v, d_o,
                     lp, plane_bytes, dv_out, dk_out, chunk_elems, s.S, Sp, s.Hl, s.Hkl, n_rep,
                     kvheads_total, ktiles, ck.n, ck.T, c, s.scale);
  if (ck.n > 1) {
    const uint32_t row_quads = (uint32_t)(s.Hkl * D / 4);
    const uint32_t seq_quads = (uint32_t)s.S * row_quads;
    const dim3 rg((seq_quads + kPreThreads - 1) / kPreThreads, (unsigned)s.b);
    const FastDiv by_rq = FastDiv::make(row_quads);
    hipLaunchKernelGGL(bwd_reduce_kernel, rg, dim3(kPreThreads), 0, stream, dv_part, dv,
                       row_quads, by_rq, seq_quads, chunk_elems, D, ck.n, ck.T);
    hipLaunchKernelGGL(bwd_reduce_kernel, rg, dim3(kPreThreads), 0, stream, dk_part, dk,
                       row_quads, by_rq, seq_quads, chunk_elems, D, ck.n, ck.T);
  }

  const int qtiles = (s.S + kDQM - 1) / kDQM;
  const int heads_total = s.b * s.Hl;
  hipLaunchKernelGGL((bwd_dq_kernel<D, SH>), dim3((unsigned)(qtiles * heads_total)),
                     dim3(kDqThreads), 0, stream, q, k, v, d_o, lp, np, dq, s.S, Sp, s.Hl,
                     n_rep, heads_total, qtiles, c, s.scale);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_bwd(const RowView &q, const RowView &k, const RowView &v,
                           const RowView &o, const float *lse, const RowView &d_o,
                           const RowView &dq, const RowView &dk, const RowView &dv,
                           void *workspace, const AttnShape &s, bool sharded,
                           hipStream_t stream) {
  if ((long long)s.b * s.S == 0) return hipSuccess;
  float *ws = static_cast<float *>(workspace);
  auto by_dim = [&](auto sh) {
    constexpr bool SH = decltype(sh)::value;
    switch (s.d) {
      case 64: return launch_bwd_d<64, SH>(q, k, v, o, lse, d_o, dq, dk, dv, ws, s, stream);
      case 80: return launch_bwd_d<80, SH>(q, k, v, o, lse, d_o, dq, dk, dv, ws, s, stream);
      case 96: return launch_bwd_d<96, SH>(q, k, v, o, lse, d_o, dq, dk, dv, ws, s, stream);
      default: return launch_bwd_d<128, SH>(q, k, v, o, lse, d_o, dq, dk, dv, ws, s, stream);
    }
  };
  return sharded ? by_dim(std::true_type{}) : by_dim(std::false_type{});
}

}  // namespace basp
