// basp_attn_fwd.hip -- causal GQA attention forward for the rank's heads.
//
// Computes the scaled dot-product attention of Sec. II-A of the paper over
// the full sequence, masked causally (key j visible to query i iff j <= i),
// for each local query head h with local kv head h / n_rep:
//   O_i = sum_j softmax_j(scale * q_i . k_j) v_j,   LSE_i = log sum_j exp(.)
// The S x S score matrix is never stored: keys are visited in tiles with a
// running row maximum and row sum (online softmax), a re-association that
// changes only rounding.
//
// gfx950 mapping
//   * workgroup = 8 waves = 256 query rows of one (sequence, head), one
//     workgroup per CU (two waves per SIMD); wave w owns rows q0 + 32w .. +31,
//     one row per lane pair (l, l+32).
//   * scores are formed transposed, S^T = K Q^T, with
//     v_mfma_f32_32x32x16_bf16: K (A operand) from LDS, Q (B operand) kept
//     in registers for the whole loop.  The 32x32 accumulator then gives each
//     lane one query row and 16 keys, so the softmax statistics are lane-local
//     up to one exchange with the partner lane l^32.
//   * O^T = V^T P^T: P goes from the score accumulator straight into the B
//     operand (bf16, round to nearest even).  V^T (A operand) is read from the
//     row-major V tile with ds_read_b64_tr_b16, two 4-key reads per operand,
//     in exactly the key order the accumulator holds P in.
//   * K/V tiles of 64 keys are copied HBM -> LDS by buffer loads that write
//     LDS directly (no register staging; rows past S arrive as zeros) into a
//     ring of four stages.  Tiles are stored row-major with an XOR swizzle
//     that is conflict-free for both read patterns.  Each wave waits only for
//     its own copies of the tile it needs next, passes a fence-free barrier,
//     and then issues the copies of the tile three ahead into the stage every
//     wave has just finished with, so two later tiles stay in flight.
//   * tiles left of the diagonal band are software-pipelined inside each
//     wave: the score products of tile t+1 are issued between the
//     exponentials of tile t, and the row sum of t and row maxima of t+1
//     between the P V products of t, one product per slot with its operand
//     read two slots ahead.  Every stretch of a wave's instruction stream
//     thus mixes matrix and vector work; the arithmetic and its order per
//     tile are unchanged (bit-identical results).
//   * LDS holds the K tiles of the four ring stages, then their V tiles, and
//     the pipelined loop is unrolled over the four stages: every operand
//     address is a lane's fixed offset plus an instruction immediate, with
//     no per-tile address arithmetic.
//   * the running maximum used as the exponent reference only moves when a
//     row's maximum grows by more than 8 (in log2 units): P <= 2^8 stays exact
//     in bf16's relative precision and O is rescaled only on those tiles.
//   * tiles strictly below the workgroup's diagonal band run a loop without
//     any masking code; band tiles are masked, and a wave skips band tiles
//     past its last row.  The grid is one-dimensional, heaviest query tiles
//     first, heads fastest, so heads sharing a kv head run side by side.
//   * in the diagonal band a wave raises its issue priority over the score
//     products, so the two waves of a SIMD drift apart: one's softmax
//     overlaps the other's MFMAs.
//   * tensors are read and written through row views: the local
//     head-sharded tensors, or (SH) the G sequence shards of the exchange in
//     place, whose row counts are multiples of 256 so that a workgroup's
//     rows and a key tile each lie in one shard; K/V tiles then take the
//     buffer of their own rows.
#include <math.h>

#include <type_traits>

#include "basp_device.hpp"
#include "basp_internal.hpp"

namespace basp {
namespace {

constexpr int kThreads = 512;
constexpr int kWaves = 8;
constexpr int kBM = 32 * kWaves;   // query rows per workgroup
constexpr int kStages = 4;
constexpr int kPD = 2;            // tiles in flight behind the one being read
constexpr int kBN = 64;           // keys per tile
constexpr float kRescaleSlack = 8.f;  // log2 headroom before the reference max moves
// Instruction classes of __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedValu = 0x002;
constexpr int kSchedMfma = 0x008;
constexpr int kSchedDsRead = 0x100;

template <int D>
struct FwdCfg {
  static constexpr int DC = HeadDim<D>::DC;  // computed width (columns past D are zero)
  static constexpr int LW = HeadDim<D>::LW;  // LDS row layout
  static constexpr int TILE_BYTES = kBN * LW * 2;
  static constexpr int STAGE_BYTES = 2 * TILE_BYTES;  // K, V
  static constexpr int NS = DC / 16;                  // 16-deep steps over the head dim
  static constexpr int NE = DC / 32;                  // 32-wide head-dim subtiles of O
  static constexpr int CPR = LW / 8;                  // 16-byte chunk slots per LDS row
  static constexpr int DMA_PER_WAVE = kBN * CPR / kThreads;  // 1 KB loads per wave per tensor
};

template <int D, bool SH>
__global__ __launch_bounds__(kThreads, 1) void attn_fwd_kernel(
    const RowView qv, const RowView kv, const RowView vv, const RowView ov,
    float *__restrict__ lse, int S, int Hl, int n_rep, int heads_total, int qtiles,
    float c /* scale * log2(e) */) {
  using C = FwdCfg<D>;
  using T = LdsTile<C::LW>;
  // LDS: the K tiles of the kStages ring stages, then their V tiles, so that
  // a stage's K and V tiles sit at the same offset from two fixed bases.
  __shared__ __attribute__((aligned(16))) unsigned char smem[kStages * C::STAGE_BYTES];
  constexpr int kVRegion = kStages * C::TILE_BYTES;

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave index, held in an SGPR
  const int l32 = lane & 31, hh = lane >> 5;

  const int L = blockIdx.x;
  const int qt = qtiles - 1 - L / heads_total;
  const int hb = L % heads_total;
  const int beta = hb / Hl, h = hb % Hl, kvh = h / n_rep;
  const int q0 = qt * kBM;
  const int wrow0 = q0 + 32 * w;
  const int row = wrow0 + l32;

  const uint32_t q_row_bytes = qv.row_elems * 2, kv_row_bytes = kv.row_elems * 2;
  uint32_t q_left, kv_left;
  // Q of rows q0 .. (rows past the buffer's end read as zeros)
  const rsrc_t rq =
      make_rsrc(view_row<SH, const uint16_t>(qv, beta, q0, h, D, q_left), q_left * q_row_bytes);
  // Local K/V: one resource per head for every tile.  Sharded: one per shard.
  u32x4 rk = {}, rv = {};
  if constexpr (!SH) {
    rk = make_rsrc_words(view_row<false, const uint16_t>(kv, beta, 0, kvh, D, kv_left),
                         kv_left * kv_row_bytes);
    rv = make_rsrc_words(view_row<false, const uint16_t>(vv, beta, 0, kvh, D, kv_left),
                         kv_left * kv_row_bytes);
  }
  const uint32_t smem_lds = lds_addr_of(smem);

  // Q fragments (B operand of S^T = K Q^T): row `row`, e = 16s + 8hh .. +7.
  bf16x8 qf[C::NS];
#pragma unroll
  for (int s = 0; s < C::NS; ++s)
    qf[s] = 2 * s < D / 8
                ? as_bf16x8(buf_load16(rq, (uint32_t)(row - q0) * q_row_bytes + (2 * s + hh) * 16))
                : bf16x8{};  // columns past D
  // Retire the Q loads before any tile copy is in flight: the compiler does
  // not count the copies, and a wait for Q inside the tile loop would also
  // drain the prefetched tiles.
  wait_vmcnt<0>();

  const int kv_end = min(S, q0 + kBM);
  const int nt = (kv_end + kBN - 1) / kBN;

  uint32_t g_off[C::DMA_PER_WAVE];
#pragma unroll
  for (int i = 0; i < C::DMA_PER_WAVE; ++i)
    g_off[i] = dma_src_off<C::LW, D>((w * C::DMA_PER_WAVE + i) * 64 + lane, kv_row_bytes);
  // Sharded: tiles are loaded in order, so the resources move to the next
  // shard only when the tiles of the current one are used up.
  uint32_t sh_tiles = 0, sh_base = 0;
  auto load_tile = [&](int t) {  // issue; lands asynchronously in stage t % kStages
    const uint32_t ks = smem_lds + (t % kStages) * C::TILE_BYTES;
    uint32_t base = (uint32_t)(t * kBN) * kv_row_bytes;
    if constexpr (SH) {
      if (sh_tiles == 0) {  // wave-uniform; tile t is the first of its shard
        uint32_t left;
        rk = make_rsrc_words(view_row<true, const uint16_t>(kv, beta, t * kBN, kvh, D, left),
                             left * kv_row_bytes);
        rv = make_rsrc_words(view_row<true, const uint16_t>(vv, beta, t * kBN, kvh, D, left),
                             left * kv_row_bytes);
        sh_tiles = left / kBN;
        sh_base = 0;
      }
      base = sh_base;
      sh_base += kBN * kv_row_bytes;
      --sh_tiles;
    }
#pragma unroll
    for (int i = 0; i < C::DMA_PER_WAVE; ++i) {
      const uint32_t lds_off = ks + (w * C::DMA_PER_WAVE + i) * 1024;
      buf_load16_lds_async(rk, base + g_off[i], lds_off);
      buf_load16_lds_async(rv, base + g_off[i], lds_off + kVRegion);
    }
  };
  // Wait until this wave's loads of tile t landed, with `ahead` later tiles
  // (2 * DMA_PER_WAVE loads each) still in flight.
  auto wait_tile = [&](int ahead) {
    if (ahead >= 2) wait_vmcnt<4 * C::DMA_PER_WAVE>();
    else if (ahead == 1) wait_vmcnt<2 * C::DMA_PER_WAVE>();
    else wait_vmcnt<0>();
  };

  // LDS offsets of this lane's operand reads (fixed across tiles).
  // A of S^T: K row 32m + l32, chunk 2s + hh.  The swizzle depends on the
  // row modulo 16 only, so row 32 + r sits 32 rows further on.
  int k_off[C::NS];
#pragma unroll
  for (int s = 0; s < C::NS; ++s) {
    k_off[s] = T::off(l32, 2 * s + hh);
    asm volatile("" : "+v"(k_off[s]));  // keep in a register, do not recompute per tile
  }
  // A of O^T: V^T rows e = 32n + l32, keys 16*s2 + 4hh + {0..3} and + 8.
  // Transposed A operand: rows 16*s2 + 4hh (+8), columns 32n + 16*((lane/16)&1);
  // row block s2 sits 16*s2 rows further on (same swizzle).
  int v_off[C::NE][2];
#pragma unroll
  for (int n = 0; n < C::NE; ++n)
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      v_off[n][x] =
          kVRegion + tr_piece_off<C::LW>(4 * hh + 8 * x, 32 * n + 16 * ((lane >> 4) & 1), lane);
      asm volatile("" : "+v"(v_off[n][x]));
    }

  f32x16 oacc[C::NE];
#pragma unroll
  for (int n = 0; n < C::NE; ++n)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[n][r] = 0.f;
  float m_ref = -INFINITY, l_run = 0.f;

  for (int t = 0; t <= kPD && t < nt; ++t) load_tile(t);

  // One tile: scores, softmax update, P V.  MASK only for tiles that can
  // hold keys past some row of the workgroup (the diagonal band).
  auto tile = [&](int t, auto mask_tag) {
    constexpr bool MASK = decltype(mask_tag)::value;
    const int j0 = t * kBN;
    const unsigned char *Ks = smem + (t % kStages) * C::TILE_BYTES;
    const unsigned char *Vs = Ks;  // v_off holds the V region's base

    wave_priority<1>();  // the score products run ahead of the partner wave's softmax
    f32x16 sacc[2];
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      const bf16x8 a = *reinterpret_cast<const bf16x8 *>(Ks + k_off[0] + m * 32 * T::ROW_BYTES);
      sacc[m] = mfma32x32x16(a, qf[0], f32x16{});
    }
#pragma unroll
    for (int s = 1; s < C::NS; ++s)
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        const bf16x8 a = *reinterpret_cast<const bf16x8 *>(Ks + k_off[s] + m * 32 * T::ROW_BYTES);
        sacc[m] = mfma32x32x16(a, qf[s], sacc[m]);
      }
    // Schedule: LDS reads run one k-step ahead of the MFMAs.
    __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 4, 0);
#pragma unroll
    for (int i = 0; i < C::NS - 2; ++i) {
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, 2, 0);
      __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(kSchedMfma, 4, 0);
    wave_priority<0>();

    // sacc[m][r] = S^T[key j0 + 32m + 8(r/4) + 4hh + r%4][query row]
    if constexpr (MASK) {
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j = j0 + 32 * m + 8 * (r >> 2) + 4 * hh + (r & 3);
          if (j > row) sacc[m][r] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[m][r]);
    mx = pair_max(mx) * c;
    // Move the reference only when the row maximum outgrew it by the slack
    // (always on a row's first tile, where m_ref is -inf).
    const bool grow = mx > m_ref + kRescaleSlack;
    if (__builtin_amdgcn_ballot_w64(grow)) {  // wave-uniform, rare after the first tiles
      asm volatile("" ::: "memory");  // keep this a real branch (no if-conversion)
      const float m_new = grow ? mx : m_ref;
      const float alpha = fast_exp2(m_ref - m_new);
      m_ref = m_new;
      l_run *= alpha;
#pragma unroll
      for (int n = 0; n < C::NE; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[n][r] *= alpha;
    }
    float psum = 0.f;
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = fast_exp2(fmaf(sacc[m][r], c, -m_ref));
        sacc[m][r] = p;
        psum += p;
      }
    l_run += psum;

    bf16x8 pf[kBN / 16];
#pragma unroll
    for (int s2 = 0; s2 < kBN / 16; ++s2) {
      const int m = s2 >> 1, b8 = (s2 & 1) * 8;
      u32x4 t4 = {pack_bf16x2(sacc[m][b8 + 0], sacc[m][b8 + 1]),
                  pack_bf16x2(sacc[m][b8 + 2], sacc[m][b8 + 3]),
                  pack_bf16x2(sacc[m][b8 + 4], sacc[m][b8 + 5]),
                  pack_bf16x2(sacc[m][b8 + 6], sacc[m][b8 + 7])};
      pf[s2] = as_bf16x8(t4);
    }
#pragma unroll
    for (int n = 0; n < C::NE; ++n)
#pragma unroll
      for (int s2 = 0; s2 < kBN / 16; ++s2) {
        const bf16x8 a = tr_operand(Vs, v_off[n][0] + s2 * 16 * T::ROW_BYTES,
                                    v_off[n][1] + s2 * 16 * T::ROW_BYTES);
        oacc[n] = mfma32x32x16(a, pf[s2], oacc[n]);
      }
    // Schedule: transposed reads run two operands ahead of the MFMAs.
    __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 4, 0);
#pragma unroll
    for (int i = 0; i < C::NE * (kBN / 16) - 2; ++i) {
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
      __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(kSchedMfma, 2, 0);
  };
  // Ring discipline: tiles 0 .. kPD are issued up front, then iteration t
  // (of either loop below) issues tile t + kPD + 1 into the stage of tile
  // t - 1, after a barrier that every wave passes only once it has finished
  // with tile t - 1.  Before the barrier a wave waits for its own copies of
  // the tile it is about to read, with `ahead` later tiles left in flight.
  auto make_visible = [&](int ahead, int issue) __attribute__((always_inline)) {
    wait_tile(ahead);
    barrier_no_fence();
    if (issue < nt) load_tile(issue);
  };

  // Tiles before t_mask need no mask.  They run software-pipelined: while
  // the softmax of tile t (exponentials, conversions, row sum) is computed,
  // the score products of tile t+1 are issued, and while P V of tile t runs,
  // the row maxima of tile t+1 are formed, so that every stretch of the
  // wave's instruction stream mixes matrix and vector work.  The arithmetic
  // and its order per tile are those of `tile`: bit-identical results.
  const int t_mask = min(nt, q0 / kBN);
  auto scores = [&](int t, f32x16 (&sc)[2]) __attribute__((always_inline)) {
    const unsigned char *Ks = smem + (t % kStages) * C::TILE_BYTES;
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      const bf16x8 a = *reinterpret_cast<const bf16x8 *>(Ks + k_off[0] + m * 32 * T::ROW_BYTES);
      sc[m] = mfma32x32x16(a, qf[0], f32x16{});
    }
#pragma unroll
    for (int s2 = 1; s2 < C::NS; ++s2)
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        const bf16x8 a = *reinterpret_cast<const bf16x8 *>(Ks + k_off[s2] + m * 32 * T::ROW_BYTES);
        sc[m] = mfma32x32x16(a, qf[s2], sc[m]);
      }
  };
  auto row_max = [&](const f32x16 (&sc)[2]) __attribute__((always_inline)) {
    float mx = -INFINITY;
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[m][r]);
    return pair_max(mx) * c;
  };
  auto move_reference = [&](float mx) __attribute__((always_inline)) {
    const bool grow = mx > m_ref + kRescaleSlack;
    if (__builtin_amdgcn_ballot_w64(grow)) {  // wave-uniform, rare after the first tiles
      asm volatile("" ::: "memory");
      const float m_new = grow ? mx : m_ref;
      const float alpha = fast_exp2(m_ref - m_new);
      m_ref = m_new;
      l_run *= alpha;
#pragma unroll
      for (int n = 0; n < C::NE; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[n][r] *= alpha;
    }
  };
  auto exps = [&](f32x16 (&sc)[2], bf16x8 (&pf)[kBN / 16]) __attribute__((always_inline)) {
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[m][r] = fast_exp2(fmaf(sc[m][r], c, -m_ref));
#pragma unroll
    for (int s2 = 0; s2 < kBN / 16; ++s2) {
      const int m = s2 >> 1, b8 = (s2 & 1) * 8;
      pf[s2] = as_bf16x8(u32x4{pack_bf16x2(sc[m][b8 + 0], sc[m][b8 + 1]),
                               pack_bf16x2(sc[m][b8 + 2], sc[m][b8 + 3]),
                               pack_bf16x2(sc[m][b8 + 4], sc[m][b8 + 5]),
                               pack_bf16x2(sc[m][b8 + 6], sc[m][b8 + 7])});
    }
  };
  auto row_sum = [&](const f32x16 (&sc)[2]) __attribute__((always_inline)) {
    float psum = 0.f;
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int r = 0; r < 16; ++r) psum += sc[m][r];
    l_run += psum;
  };
  auto pv = [&](int t, const bf16x8 (&pf)[kBN / 16]) __attribute__((always_inline)) {
    const unsigned char *Vs = smem + (t % kStages) * C::TILE_BYTES;
#pragma unroll
    for (int n = 0; n < C::NE; ++n)
#pragma unroll
      for (int s2 = 0; s2 < kBN / 16; ++s2) {
        const bf16x8 a = tr_operand(Vs, v_off[n][0] + s2 * 16 * T::ROW_BYTES,
                                    v_off[n][1] + s2 * 16 * T::ROW_BYTES);
        oacc[n] = mfma32x32x16(a, pf[s2], oacc[n]);
      }
  };
  // Iteration t of the pipelined loop, tile t+1 unmasked: `cur` holds the
  // scores of tile t (reference already moved for them); the scores of tile
  // t+1 go to `nxt`.  Each block is a sequence of slots of one product each,
  // fenced by scheduling barriers: the slot's share of the vector work, and
  // the operand read for the product kPf slots later.
  constexpr int kPf = 2;
  auto pipelined = [&](int t, auto stage_tag, f32x16 (&cur)[2], f32x16 (&nxt)[2])
                       __attribute__((always_inline)) {
    constexpr int ST = decltype(stage_tag)::value;  // t % kStages
    make_visible(min(1, nt - 2 - t), t + kPD + 1);  // tile t+1 readable, t+2 in flight
    asm volatile("" : "+v"(m_ref));  // keep the exponent arguments here
    bf16x8 pf[kBN / 16];
    // Block X: scores of tile t+1 (16 products), exponentials of tile t, at
    // raised issue priority: of the two waves of a SIMD, the one in this
    // block keeps the matrix unit while the other is in block Y.
    wave_priority<1>();
    {
      constexpr int NG = 2 * C::NS;
      const unsigned char *Ks = smem + ((ST + 1) % kStages) * C::TILE_BYTES;
      bf16x8 op[NG];
      auto read = [&](int g) __attribute__((always_inline)) {
        op[g] = *reinterpret_cast<const bf16x8 *>(Ks + k_off[g / 2] + (g % 2) * 32 * T::ROW_BYTES);
      };
#pragma unroll
      for (int g = 0; g < kPf; ++g) read(g);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        if (g + kPf < NG) read(g + kPf);
        const int m = g % 2, s2 = g / 2;
        nxt[m] = mfma32x32x16(op[g], qf[s2], s2 == 0 ? f32x16{} : nxt[m]);
        // 32 exponentials over the 16 slots; each full group of 8 converted
#pragma unroll
        for (int e = 32 * g / NG; e < 32 * (g + 1) / NG; ++e) {
          const int mm = e / 16, r = e % 16;
          cur[mm][r] = fast_exp2(fmaf(cur[mm][r], c, -m_ref));
          if (r % 8 == 7) {
            const int b8 = r - 7;
            pf[2 * mm + b8 / 8] = as_bf16x8(u32x4{pack_bf16x2(cur[mm][b8 + 0], cur[mm][b8 + 1]),
                                                  pack_bf16x2(cur[mm][b8 + 2], cur[mm][b8 + 3]),
                                                  pack_bf16x2(cur[mm][b8 + 4], cur[mm][b8 + 5]),
                                                  pack_bf16x2(cur[mm][b8 + 6], cur[mm][b8 + 7])});
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    wave_priority<0>();
    // Block Y: P V of tile t (16 products), row sum of t, row maxima of t+1.
    float psum = 0.f, mx = -INFINITY;
    {
      constexpr int NG = C::NE * (kBN / 16);
      const unsigned char *Vs = smem + ST * C::TILE_BYTES;
      bf16x8 op[NG];
      auto read = [&](int g) __attribute__((always_inline)) {
        const int n = g / (kBN / 16), s2 = g % (kBN / 16);
        op[g] = tr_operand(Vs, v_off[n][0] + s2 * 16 * T::ROW_BYTES,
                           v_off[n][1] + s2 * 16 * T::ROW_BYTES);
      };
#pragma unroll
      for (int g = 0; g < kPf; ++g) read(g);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        if (g + kPf < NG) read(g + kPf);
        const int n = g / (kBN / 16), s2 = g % (kBN / 16);
        oacc[n] = mfma32x32x16(op[g], pf[s2], oacc[n]);
#pragma unroll
        for (int e = 32 * g / NG; e < 32 * (g + 1) / NG; ++e) psum += cur[e / 16][e % 16];
#pragma unroll
        for (int e = 32 * g / NG; e < 32 * (g + 1) / NG; ++e) mx = fmaxf(mx, nxt[e / 16][e % 16]);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    l_run += psum;
    move_reference(pair_max(mx) * c);  // after P V of tile t, before the exponentials of t+1
  };
  // The last unmasked tile t: no scores to start.
  auto pipelined_last = [&](int t, f32x16 (&cur)[2]) __attribute__((always_inline)) {
    make_visible(min(1, nt - 2 - t), t + kPD + 1);  // tile t+1 (the first masked one)
    asm volatile("" : "+v"(m_ref));
    bf16x8 pf[kBN / 16];
    exps(cur, pf);
    __builtin_amdgcn_sched_barrier(0);
    pv(t, pf);
    row_sum(cur);
    __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 4, 0);
#pragma unroll
    for (int i = 0; i < C::NE * (kBN / 16) - 2; ++i) {
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
      __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 0);
      __builtin_amdgcn_sched_group_barrier(kSchedValu, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(kSchedMfma, 2, 0);
    __builtin_amdgcn_sched_barrier(0);
  };
  if (t_mask > 0) {
    f32x16 sa[2], sb[2];
    make_visible(min(kPD, nt - 1), nt);  // tile 0; tile kPD + 1 is issued by iteration 0
    scores(0, sa);
    move_reference(row_max(sa));
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using I3 = std::integral_constant<int, 3>;
    static_assert(kStages == 4, "the unrolled loop assumes four ring stages");
    int t = 0;
    for (; t + 4 < t_mask; t += 4) {  // t % 4 == 0: every stage offset a constant
      pipelined(t, I0{}, sa, sb);
      pipelined(t + 1, I1{}, sb, sa);
      pipelined(t + 2, I2{}, sa, sb);
      pipelined(t + 3, I3{}, sb, sa);
    }
    // 1 to 4 unmasked tiles left, the last of them without scores to start
    if (t + 1 < t_mask) {
      pipelined(t, I0{}, sa, sb);
      if (t + 2 < t_mask) {
        pipelined(t + 1, I1{}, sb, sa);
        if (t + 3 < t_mask) {
          pipelined(t + 2, I2{}, sa, sb);
          pipelined_last(t + 3, sb);
        } else {
          pipelined_last(t + 2, sa);
        }
      } else {
        pipelined_last(t + 1, sb);
      }
    } else {
      pipelined_last(t, sa);
    }
  }
  for (int t = t_mask; t < nt; ++t) {  // the diagonal band, masked
    make_visible(min(kPD, nt - 1 - t), t + kPD + 1);
    if (t * kBN <= wrow0 + 31) tile(t, std::true_type{});  // wave-uniform
  }

  // oacc[n][r] = O^T[e = 32n + 8(r/4) + 4hh + r%4][query row] (unnormalised)
  const float l_tot = pair_sum(l_run);
  if (row < S) {
    const float inv = 1.f / l_tot;
    uint32_t o_left;
    uint16_t *ob = view_row<SH, uint16_t>(ov, beta, q0, h, D, o_left) +
                   (size_t)(row - q0) * ov.row_elems;
#pragma unroll
    for (int n = 0; n < C::NE; ++n)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        if (32 * n + 8 * g >= D) continue;  // padding columns
        u32x2 val = {pack_bf16x2(oacc[n][4 * g] * inv, oacc[n][4 * g + 1] * inv),
                     pack_bf16x2(oacc[n][4 * g + 2] * inv, oacc[n][4 * g + 3] * inv)};
        *reinterpret_cast<u32x2 *>(ob + 32 * n + 8 * g + 4 * hh) = val;
      }
    if (hh == 0)
      lse[((size_t)beta * Hl + h) * S + row] = (m_ref + fast_log2(l_tot)) * 0.69314718055994531f;
  }
}

}  // namespace

hipError_t launch_attn_fwd(const RowView &q, const RowView &k, const RowView &v,
                           const RowView &o, float *lse, const AttnShape &s, bool sharded,
                           hipStream_t stream) {
  const int qtiles = (s.S + kBM - 1) / kBM;
  const int heads_total = s.b * s.Hl;
  const long long blocks = (long long)qtiles * heads_total;
  if (blocks == 0) return hipSuccess;
  const float c = s.scale * 1.4426950408889634f;
  const int n_rep = s.Hl / s.Hkl;
  auto go = [&](auto kernel) {
    hipLaunchKernelGGL(kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream, q, k, v, o, lse,
                       s.S, s.Hl, n_rep, heads_total, qtiles, c);
  };
  auto by_dim = [&](auto sh) {
    constexpr bool SH = decltype(sh)::value;
    switch (s.d) {
      case 64: go(attn_fwd_kernel<64, SH>); break;
      case 80: go(attn_fwd_kernel<80, SH>); break;
      case 96: go(attn_fwd_kernel<96, SH>); break;
      default: go(attn_fwd_kernel<128, SH>); break;
    }
  };
  if (sharded)
    by_dim(std::true_type{});
  else
    by_dim(std::false_type{});
  return hipGetLastError();
}

}  // namespace basp
