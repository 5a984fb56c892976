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
// Four kernels, all deterministic (no atomics):
//   bwd_pre   D for every (sequence, head, row)
//   bwd_kv    key-stationary, twice (dV, then dK): a workgroup owns 128
//             keys of one kv head and sweeps every query row at or after
//             them, for all query heads of the GQA group, accumulating in
//             registers
//   bwd_dq    query-stationary: like the forward, a workgroup owns 128 rows
//             of one query head and sweeps the keys up to the diagonal
// On gfx950 both main kernels use v_mfma_f32_32x32x16_bf16 with fp32
// accumulation.  Which operand order is used is chosen so that every
// elementwise step (P, dS) happens in the accumulator layout and feeds the
// next product without a round trip through LDS.  Operands that must be read
// along the sequence (Q^T, dO^T, K^T) come from the same row-major LDS tiles
// through ds_read_b64_tr_b16, in the order the accumulator holds P and dS.
// Tiles are filled with 16-byte buffer loads (rows past S read as zero),
// double-buffered, and each 64-wide tile is processed in two 32-wide halves.
#include <math.h>

#include "basp_device.hpp"
#include "basp_internal.hpp"

namespace basp {
namespace {

constexpr int kThreads = 256;
constexpr float kLog2e = 1.4426950408889634f;

// Row chunking of the key-stationary kernels: 1 chunk up to 2048 rows, 2 up
// to 8192, else 4 (multiples of 64 rows), enough workgroups to balance the
// causal triangle over the GPU.  Workspace: D, then (if chunked) the dV and dK
// partial sums [chunk][b][S][H_kv/G][d].
struct BwdChunks {
  int n, rows;
  size_t part_offset_floats;
};

BwdChunks bwd_chunks(const AttnShape &s) {
  BwdChunks ck;
  ck.n = s.S <= 2048 ? 1 : (s.S <= 8192 ? 2 : 4);
  ck.rows = ((s.S + ck.n - 1) / ck.n + 63) / 64 * 64;
  ck.n = (s.S + ck.rows - 1) / ck.rows;
  if (ck.n < 1) ck.n = 1;
  const size_t d_floats = (size_t)s.b * s.Hl * s.S;
  ck.part_offset_floats = (d_floats + 63) & ~(size_t)63;  // 256-byte aligned
  return ck;
}

// ---------------------------------------------------------------- bwd_pre
// One group of D/8 lanes per (beta, row, head); 16-byte loads of O and dO.
template <int D>
__global__ __launch_bounds__(kThreads) void bwd_pre_kernel(
    const uint16_t *__restrict__ o, const uint16_t *__restrict__ d_o,
    float *__restrict__ Dbuf, long long rows /* b*S*Hl */, int S, int Hl) {
  constexpr int LPR = D / 8;  // lanes per row
  const long long gid = (long long)blockIdx.x * kThreads + threadIdx.x;
  const long long r = gid / LPR;
  const int sub = (int)(gid % LPR);
  float acc = 0.f;
  if (r < rows) {
    const u32x4 a = reinterpret_cast<const u32x4 *>(o + r * D)[sub];
    const u32x4 b = reinterpret_cast<const u32x4 *>(d_o + r * D)[sub];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc += bf16_bits_to_f32(a[i] & 0xFFFFu) * bf16_bits_to_f32(b[i] & 0xFFFFu);
      acc += bf16_bits_to_f32(a[i] >> 16) * bf16_bits_to_f32(b[i] >> 16);
    }
  }
#pragma unroll
  for (int off = LPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
  if (r < rows && sub == 0) {
    // r = (beta*S + i)*Hl + h  ->  D[beta][h][i]
    const long long bi = r / Hl;
    const int h = (int)(r - bi * Hl);
    const long long beta = bi / S;
    const int i = (int)(bi - beta * S);
    Dbuf[(beta * Hl + h) * S + i] = acc;
  }
}

// ------------------------------------------------------ bwd_dv / bwd_dk
// Key-stationary.  A workgroup of 4 waves owns 128 keys of one kv head (32
// per wave) and sweeps every 64-row query tile at or after them, for all
// query heads of the GQA group.  Two instances of one kernel:
//   kDV: S = Q K^T, P = exp2(S c - LSE2),   dV^T += dO^T P
//   kDK: S, dP = dO V^T, dS = P (dP - D),   dK^T += Q^T dS
// Keeping dV and dK in separate launches recomputes S once more, but leaves
// every wave independent (no exchange between waves, one barrier per step)
// and small enough for two waves per SIMD.
constexpr int kKN = 128;  // keys per workgroup (32 per wave)
constexpr int kQM = 64;   // query rows per step (two 32-row halves)
enum KvGrad { kDV = 0, kDK = 1 };

template <int D>
struct KvCfg {
  static constexpr int TILE_BYTES = kQM * D * 2;
  // Q tile, dO tile, then 2 x kQM floats (LSE in log2 units, D).
  static constexpr int STAGE_BYTES = 2 * TILE_BYTES + 2 * kQM * 4;
  static constexpr int NS = D / 16;
  static constexpr int NE = D / 32;
  static constexpr int CPR = D / 8;
  static constexpr int CHUNKS = kQM * CPR / kThreads;
};

template <int D, int G>
__global__ __launch_bounds__(kThreads, 2) void bwd_kv_kernel(
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k,
    const uint16_t *__restrict__ v, const uint16_t *__restrict__ d_o,
    const float *__restrict__ lse, const float *__restrict__ Dbuf,
    float *__restrict__ out, int S, int Hl, int Hkl, int n_rep, int kvheads_total,
    int ktiles, int chunk_rows, float c /* scale*log2e */, float out_scale) {
  using C = KvCfg<D>;
  using T = LdsTile<D>;
  __shared__ __attribute__((aligned(16))) unsigned char smem[2 * C::STAGE_BYTES];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  // Work item: (row chunk ch, key tile kt, sequence x kv head hb).  The rows a
  // key tile needs, [k0, S), are cut at multiples of chunk_rows; each chunk
  // writes its own partial sum (slice ch of `out`), so long key tiles are
  // spread over several workgroups.  Earlier key tiles come first within a
  // chunk (they have more rows).
  const int L = blockIdx.x;
  const int hb = L % kvheads_total;
  const int kt = (L / kvheads_total) % ktiles;
  const int ch = L / (kvheads_total * ktiles);
  const int beta = hb / Hkl, kvh = hb % Hkl;
  const int k0 = kt * kKN;
  const int r_lo = max(k0, ch * chunk_rows), r_hi = min(S, (ch + 1) * chunk_rows);
  if (r_lo >= r_hi) return;  // workgroup-uniform: this chunk lies before the keys
  const int wk0 = k0 + 32 * w;
  const int key = wk0 + l32;

  const uint32_t q_row_bytes = (uint32_t)Hl * D * 2, kv_row_bytes = (uint32_t)Hkl * D * 2;
  const size_t kvoff = ((size_t)beta * S * Hkl + kvh) * D;
  out += (size_t)ch * ((size_t)kvheads_total * S * D);
  // K (and V for dK) of this lane's key as B operands (B[e][j] = K[j][e]).
  bf16x8 kf[C::NS], vf[G == kDK ? C::NS : 1];
  {
    const rsrc_t rk = make_rsrc(k + kvoff, (uint32_t)S * kv_row_bytes);
#pragma unroll
    for (int s = 0; s < C::NS; ++s)
      kf[s] = as_bf16x8(buf_load16(rk, (uint32_t)key * kv_row_bytes + (2 * s + hh) * 16));
    if constexpr (G == kDK) {
      const rsrc_t rv = make_rsrc(v + kvoff, (uint32_t)S * kv_row_bytes);
#pragma unroll
      for (int s = 0; s < C::NS; ++s)
        vf[s] = as_bf16x8(buf_load16(rv, (uint32_t)key * kv_row_bytes + (2 * s + hh) * 16));
    }
  }

  f32x16 acc[C::NE];
#pragma unroll
  for (int n = 0; n < C::NE; ++n)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[n][r] = 0.f;

  const int steps_per_head = (r_hi - r_lo + kQM - 1) / kQM;
  const int nsteps = steps_per_head * n_rep;

  uint32_t g_off[C::CHUNKS];
  int s_off[C::CHUNKS];
#pragma unroll
  for (int r = 0; r < C::CHUNKS; ++r) {
    const int cidx = tid + r * kThreads;
    const int ir = cidx / C::CPR, cc = cidx % C::CPR;
    g_off[r] = (uint32_t)ir * q_row_bytes + cc * 16;
    s_off[r] = T::off(ir, cc);
  }
  // A of S and dP: row l32 (+32 for the second half), chunk 2s + hh.
  int a_off[C::NS];
#pragma unroll
  for (int s = 0; s < C::NS; ++s) a_off[s] = T::off(l32, 2 * s + hh);
  // Transposed A of dV^T / dK^T: rows 16*s2 + 4hh (+8), columns 32n + 16*((lane/16)&1).
  int t_off[C::NE][2];
#pragma unroll
  for (int n = 0; n < C::NE; ++n)
#pragma unroll
    for (int x = 0; x < 2; ++x)
      t_off[n][x] = tr_piece_off<D>(4 * hh + 8 * x, 32 * n + 16 * ((lane >> 4) & 1), lane);

  u32x4 qreg[C::CHUNKS], doreg[C::CHUNKS];
  float aux = 0.f;  // LSE2 (tid < 64) or D (64 <= tid < 128) of one row

  // Rows past r_hi (in the last step of a chunk that ends before S) are
  // read as data but carry LSE = +inf, so their P is exactly zero.
  auto step_coords = [&](int st, int &h, int &i0) {
    const int hr = st / steps_per_head;
    h = kvh * n_rep + hr;
    i0 = r_lo + (st - hr * steps_per_head) * kQM;
  };

  auto load_step = [&](int st) {
    int h, i0;
    step_coords(st, h, i0);
    const size_t hoff = ((size_t)beta * S * Hl + h) * D;
    const rsrc_t rq = make_rsrc(q + hoff, (uint32_t)S * q_row_bytes);
    const rsrc_t rd = make_rsrc(d_o + hoff, (uint32_t)S * q_row_bytes);
    const uint32_t base = (uint32_t)i0 * q_row_bytes;
#pragma unroll
    for (int r = 0; r < C::CHUNKS; ++r) {
      qreg[r] = buf_load16(rq, base + g_off[r]);
      doreg[r] = buf_load16(rd, base + g_off[r]);
    }
    if (tid < 2 * kQM) {
      const int i = i0 + (tid & (kQM - 1));
      const size_t idx = ((size_t)beta * Hl + h) * S + i;
      if (tid < kQM)
        aux = i < r_hi ? lse[idx] * kLog2e : INFINITY;
      else
        aux = i < r_hi ? Dbuf[idx] : 0.f;
    }
  };

  auto store_step = [&](int buf) {
    unsigned char *Qs = smem + buf * C::STAGE_BYTES;
    unsigned char *dOs = Qs + C::TILE_BYTES;
    float *aux_s = reinterpret_cast<float *>(dOs + C::TILE_BYTES);
#pragma unroll
    for (int r = 0; r < C::CHUNKS; ++r) {
      *reinterpret_cast<u32x4 *>(Qs + s_off[r]) = qreg[r];
      *reinterpret_cast<u32x4 *>(dOs + s_off[r]) = doreg[r];
    }
    if (tid < 2 * kQM) aux_s[tid] = aux;
  };

  load_step(0);
  store_step(0);
  __syncthreads();

  for (int st = 0; st < nsteps; ++st) {
    if (st + 1 < nsteps) load_step(st + 1);
    int h_unused, i0;
    step_coords(st, h_unused, i0);
    const unsigned char *Qs = smem + (st & 1) * C::STAGE_BYTES;
    const unsigned char *dOs = Qs + C::TILE_BYTES;
    const float *lse_s = reinterpret_cast<const float *>(dOs + C::TILE_BYTES);
    const float *D_s = lse_s + kQM;
    // The transposed operand of the accumulation: dO^T for dV, Q^T for dK.
    const unsigned char *Ts = G == kDV ? dOs : Qs;

#pragma unroll
    for (int m = 0; m < 2; ++m) {
      if (i0 + 32 * m + 31 < wk0) continue;  // wave-uniform: half entirely above the keys
      // sacc[r] holds row i0 + 32m + 8(r/4) + 4hh + r%4, key `key`.
      f32x16 sacc, pacc;
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[r] = 0.f;
      if constexpr (G == kDK) {
#pragma unroll
        for (int r = 0; r < 16; ++r) pacc[r] = 0.f;
      }
#pragma unroll
      for (int s = 0; s < C::NS; ++s) {
        const bf16x8 aq = *reinterpret_cast<const bf16x8 *>(Qs + a_off[s] + m * 32 * T::ROW_BYTES);
        sacc = mfma32x32x16(aq, kf[s], sacc);
        if constexpr (G == kDK) {
          const bf16x8 ad =
              *reinterpret_cast<const bf16x8 *>(dOs + a_off[s] + m * 32 * T::ROW_BYTES);
          pacc = mfma32x32x16(ad, vf[s], pacc);
        }
      }
      // P (masked on the diagonal), then dS for dK.
      if (i0 + 32 * m < wk0 + 31) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 l4 = *reinterpret_cast<const f32x4 *>(lse_s + 32 * m + 8 * g + 4 * hh);
#pragma unroll
          for (int x = 0; x < 4; ++x) {
            const int r = 4 * g + x;
            const float p = fast_exp2(fmaf(sacc[r], c, -l4[x]));
            sacc[r] = key > i0 + 32 * m + 8 * g + 4 * hh + x ? 0.f : p;
          }
        }
      } else {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 l4 = *reinterpret_cast<const f32x4 *>(lse_s + 32 * m + 8 * g + 4 * hh);
#pragma unroll
          for (int x = 0; x < 4; ++x) sacc[4 * g + x] = fast_exp2(fmaf(sacc[4 * g + x], c, -l4[x]));
        }
      }
      if constexpr (G == kDK) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const f32x4 d4 = *reinterpret_cast<const f32x4 *>(D_s + 32 * m + 8 * g + 4 * hh);
#pragma unroll
          for (int x = 0; x < 4; ++x) sacc[4 * g + x] *= pacc[4 * g + x] - d4[x];
        }
      }
      // P or dS as the B operand along the rows: block s2 covers rows
      // 32m + 16*s2 .. +15, slot t <-> register 8*s2 + t.
      bf16x8 b[2];
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const int b8 = 8 * s2;
        u32x4 t4 = {pack_bf16x2(sacc[b8 + 0], sacc[b8 + 1]), pack_bf16x2(sacc[b8 + 2], sacc[b8 + 3]),
                    pack_bf16x2(sacc[b8 + 4], sacc[b8 + 5]), pack_bf16x2(sacc[b8 + 6], sacc[b8 + 7])};
        b[s2] = as_bf16x8(t4);
      }
      // dV^T += dO^T P  or  dK^T += Q^T dS: M = head dim, N = keys, K = rows;
      // the transposed A operand comes straight from the row-major tile.
#pragma unroll
      for (int n = 0; n < C::NE; ++n)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const int ro = (2 * m + s2) * 16 * T::ROW_BYTES;
          const bf16x8 a = tr_operand(Ts, t_off[n][0] + ro, t_off[n][1] + ro);
          acc[n] = mfma32x32x16(a, b[s2], acc[n]);
        }
    }
    if (st + 1 < nsteps) store_step((st + 1) & 1);
    __syncthreads();
  }

  // acc[n][r] = (dV or dK)^T[e = 32n + 8(r/4) + 4hh + r%4][key]
  if (key < S) {
    float *o = out + ((size_t)(beta * S + key) * Hkl + kvh) * D;
#pragma unroll
    for (int n = 0; n < C::NE; ++n)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 a = {acc[n][4 * g] * out_scale, acc[n][4 * g + 1] * out_scale,
                   acc[n][4 * g + 2] * out_scale, acc[n][4 * g + 3] * out_scale};
        *reinterpret_cast<f32x4 *>(o + 32 * n + 8 * g + 4 * hh) = a;
      }
  }
}

// ---------------------------------------------------------------- bwd_reduce
// dK or dV of a key = the sum of the partial sums of the row chunks that
// exist for its key tile, added in chunk order (deterministic).  One thread
// per 4 consecutive elements.
__global__ __launch_bounds__(kThreads) void bwd_reduce_kernel(
    const float *__restrict__ part, float *__restrict__ out, long long n4 /* b*S*Hkl*D/4 */,
    int S, int row_elems /* Hkl*D */, int nchunks, int chunk_rows) {
  const long long i4 = (long long)blockIdx.x * kThreads + threadIdx.x;
  if (i4 >= n4) return;
  const long long e = i4 * 4;
  const int key = (int)((e / row_elems) % S);
  const int first = (key / kKN) * kKN / chunk_rows;  // first chunk the key tile wrote
  const long long slice = n4 * 4;
  f32x4 acc = *reinterpret_cast<const f32x4 *>(part + (size_t)first * slice + e);
  for (int ch = first + 1; ch < nchunks; ++ch) {
    const f32x4 x = *reinterpret_cast<const f32x4 *>(part + (size_t)ch * slice + e);
    acc[0] += x[0];
    acc[1] += x[1];
    acc[2] += x[2];
    acc[3] += x[3];
  }
  *reinterpret_cast<f32x4 *>(out + e) = acc;
}

// ---------------------------------------------------------------- bwd_dq
constexpr int kDQM = 128;  // query rows per workgroup (32 per wave)
constexpr int kDQN = 64;   // keys per tile

template <int D>
struct DqCfg {
  static constexpr int TILE_BYTES = kDQN * D * 2;
  static constexpr int STAGE_BYTES = 2 * TILE_BYTES;  // K, V
  static constexpr int NS = D / 16;
  static constexpr int NE = D / 32;
  static constexpr int CPR = D / 8;
  static constexpr int CHUNKS = kDQN * CPR / kThreads;
};

template <int D>
__global__ __launch_bounds__(kThreads, 2) void bwd_dq_kernel(
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k,
    const uint16_t *__restrict__ v, const uint16_t *__restrict__ d_o,
    const float *__restrict__ lse, const float *__restrict__ Dbuf,
    float *__restrict__ dq, int S, int Hl, int Hkl, int n_rep, int heads_total,
    int qtiles, float c, float scale) {
  using C = DqCfg<D>;
  using T = LdsTile<D>;
  __shared__ __attribute__((aligned(16))) unsigned char smem[2 * C::STAGE_BYTES];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int L = blockIdx.x;
  const int qt = qtiles - 1 - L / heads_total;
  const int hb = L % heads_total;
  const int beta = hb / Hl, h = hb % Hl, kvh = h / n_rep;
  const int q0 = qt * kDQM;
  const int wrow0 = q0 + 32 * w;
  const int row = wrow0 + l32;

  const uint32_t q_row_bytes = (uint32_t)Hl * D * 2, kv_row_bytes = (uint32_t)Hkl * D * 2;
  const size_t hoff = ((size_t)beta * S * Hl + h) * D;
  const rsrc_t rq = make_rsrc(q + hoff, (uint32_t)S * q_row_bytes);
  const rsrc_t rd = make_rsrc(d_o + hoff, (uint32_t)S * q_row_bytes);
  const rsrc_t rk = make_rsrc(k + ((size_t)beta * S * Hkl + kvh) * D, (uint32_t)S * kv_row_bytes);
  const rsrc_t rv = make_rsrc(v + ((size_t)beta * S * Hkl + kvh) * D, (uint32_t)S * kv_row_bytes);

  bf16x8 qf[C::NS], df[C::NS];
#pragma unroll
  for (int s = 0; s < C::NS; ++s) {
    qf[s] = as_bf16x8(buf_load16(rq, (uint32_t)row * q_row_bytes + (2 * s + hh) * 16));
    df[s] = as_bf16x8(buf_load16(rd, (uint32_t)row * q_row_bytes + (2 * s + hh) * 16));
  }
  const size_t lidx = ((size_t)beta * Hl + h) * S + row;
  const float lse2 = row < S ? lse[lidx] * kLog2e : INFINITY;
  const float Drow = row < S ? Dbuf[lidx] : 0.f;

  const int kv_end = min(S, q0 + kDQM);
  const int nt = (kv_end + kDQN - 1) / kDQN;

  uint32_t g_off[C::CHUNKS];
  int s_off[C::CHUNKS];
#pragma unroll
  for (int r = 0; r < C::CHUNKS; ++r) {
    const int cidx = tid + r * kThreads;
    const int jr = cidx / C::CPR, cc = cidx % C::CPR;
    g_off[r] = (uint32_t)jr * kv_row_bytes + cc * 16;
    s_off[r] = T::off(jr, cc);
  }
  int a_off[C::NS];  // row l32 (+32 for m = 1), chunk 2s + hh
#pragma unroll
  for (int s = 0; s < C::NS; ++s) a_off[s] = T::off(l32, 2 * s + hh);
  // Transposed A operand: rows 16*s2 + 4hh (+8), columns 32n + 16*((lane/16)&1);
  // row block s2 sits 16*s2 rows further on (same swizzle).
  int t_off[C::NE][2];
#pragma unroll
  for (int n = 0; n < C::NE; ++n)
#pragma unroll
    for (int x = 0; x < 2; ++x)
      t_off[n][x] = tr_piece_off<D>(4 * hh + 8 * x, 32 * n + 16 * ((lane >> 4) & 1), lane);

  u32x4 kreg[C::CHUNKS], vreg[C::CHUNKS];
  auto load_tile = [&](int t) {
    const uint32_t base = (uint32_t)(t * kDQN) * kv_row_bytes;
#pragma unroll
    for (int r = 0; r < C::CHUNKS; ++r) {
      kreg[r] = buf_load16(rk, base + g_off[r]);
      vreg[r] = buf_load16(rv, base + g_off[r]);
    }
  };
  auto store_tile = [&](int buf) {
    unsigned char *Ks = smem + buf * C::STAGE_BYTES;
    unsigned char *Vs = Ks + C::TILE_BYTES;
#pragma unroll
    for (int r = 0; r < C::CHUNKS; ++r) {
      *reinterpret_cast<u32x4 *>(Ks + s_off[r]) = kreg[r];
      *reinterpret_cast<u32x4 *>(Vs + s_off[r]) = vreg[r];
    }
  };

  f32x16 qacc[C::NE];
#pragma unroll
  for (int n = 0; n < C::NE; ++n)
#pragma unroll
    for (int r = 0; r < 16; ++r) qacc[n][r] = 0.f;

  load_tile(0);
  store_tile(0);
  __syncthreads();

  for (int t = 0; t < nt; ++t) {
    if (t + 1 < nt) load_tile(t + 1);
    const int j0 = t * kDQN;
    if (j0 <= wrow0 + 31) {
      const unsigned char *Ks = smem + (t & 1) * C::STAGE_BYTES;
      const unsigned char *Vs = Ks + C::TILE_BYTES;
      // Two halves of 32 keys each (keeps the score state at 2 x 16 registers).
      // S^T = K Q^T and dP^T = V dO^T: M = 32 keys, N = this wave's rows;
      // acc[r] holds key j0 + 32m + 8(r/4) + 4hh + r%4, query row `row`.
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        if (j0 + 32 * m > wrow0 + 31) continue;  // wave-uniform: half entirely masked
        f32x16 sacc, pacc;
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[r] = pacc[r] = 0.f;
#pragma unroll
        for (int s = 0; s < C::NS; ++s) {
          const bf16x8 ak =
              *reinterpret_cast<const bf16x8 *>(Ks + a_off[s] + m * 32 * T::ROW_BYTES);
          const bf16x8 av =
              *reinterpret_cast<const bf16x8 *>(Vs + a_off[s] + m * 32 * T::ROW_BYTES);
          sacc = mfma32x32x16(ak, qf[s], sacc);
          pacc = mfma32x32x16(av, df[s], pacc);
        }
        const bool diag = j0 + 32 * m + 31 > wrow0;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float p = fast_exp2(fmaf(sacc[r], c, -lse2));
          if (diag) {
            const int j = j0 + 32 * m + 8 * (r >> 2) + 4 * hh + (r & 3);
            if (j > row) p = 0.f;
          }
          pacc[r] = p * (pacc[r] - Drow);
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
        // from the row-major K tile.
#pragma unroll
        for (int n = 0; n < C::NE; ++n)
#pragma unroll
          for (int s2 = 0; s2 < 2; ++s2) {
            const int ro = (2 * m + s2) * 16 * T::ROW_BYTES;
            const bf16x8 a = tr_operand(Ks, t_off[n][0] + ro, t_off[n][1] + ro);
            qacc[n] = mfma32x32x16(a, sb[s2], qacc[n]);
          }
      }
    }
    if (t + 1 < nt) store_tile((t + 1) & 1);
    __syncthreads();
  }

  if (row < S) {
    float *dqr = dq + ((size_t)(beta * S + row) * Hl + h) * D;
#pragma unroll
    for (int n = 0; n < C::NE; ++n)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 a = {qacc[n][4 * g] * scale, qacc[n][4 * g + 1] * scale,
                   qacc[n][4 * g + 2] * scale, qacc[n][4 * g + 3] * scale};
        *reinterpret_cast<f32x4 *>(dqr + 32 * n + 8 * g + 4 * hh) = a;
      }
  }
}

template <int D>
hipError_t launch_bwd_d(const void *q, const void *k, const void *v, const void *o,
                        const float *lse, const void *d_o, float *dq, float *dk,
                        float *dv, float *Dbuf, const AttnShape &s, hipStream_t stream) {
  auto *qp = static_cast<const uint16_t *>(q);
  auto *kp = static_cast<const uint16_t *>(k);
  auto *vp = static_cast<const uint16_t *>(v);
  auto *op = static_cast<const uint16_t *>(o);
  auto *dop = static_cast<const uint16_t *>(d_o);
  const float c = s.scale * kLog2e;
  const int n_rep = s.Hl / s.Hkl;

  const long long rows = (long long)s.b * s.S * s.Hl;
  const long long pre_threads = rows * (D / 8);
  const long long pre_blocks = (pre_threads + kThreads - 1) / kThreads;
  hipLaunchKernelGGL(bwd_pre_kernel<D>, dim3((unsigned)pre_blocks), dim3(kThreads), 0, stream,
                     op, dop, Dbuf, rows, s.S, s.Hl);

  const int ktiles = (s.S + kKN - 1) / kKN;
  const int kvheads_total = s.b * s.Hkl;
  const BwdChunks ck = bwd_chunks(s);
  const dim3 kv_grid((unsigned)(ck.n * ktiles * kvheads_total));
  float *dv_out = dv, *dk_out = dk;
  if (ck.n > 1) {  // partial sums in the workspace, reduced below
    dv_out = Dbuf + ck.part_offset_floats;
    dk_out = dv_out + (size_t)ck.n * kvheads_total * s.S * D;
  }
  hipLaunchKernelGGL((bwd_kv_kernel<D, kDV>), kv_grid, dim3(kThreads), 0, stream, qp, kp, vp,
                     dop, lse, Dbuf, dv_out, s.S, s.Hl, s.Hkl, n_rep, kvheads_total, ktiles,
                     ck.rows, c, 1.f);
  hipLaunchKernelGGL((bwd_kv_kernel<D, kDK>), kv_grid, dim3(kThreads), 0, stream, qp, kp, vp,
                     dop, lse, Dbuf, dk_out, s.S, s.Hl, s.Hkl, n_rep, kvheads_total, ktiles,
                     ck.rows, c, s.scale);
  if (ck.n > 1) {
    const long long n4 = (long long)kvheads_total * s.S * D / 4;
    const dim3 rg((unsigned)((n4 + kThreads - 1) / kThreads));
    hipLaunchKernelGGL(bwd_reduce_kernel, rg, dim3(kThreads), 0, stream, dv_out, dv, n4, s.S,
                       s.Hkl * D, ck.n, ck.rows);
    hipLaunchKernelGGL(bwd_reduce_kernel, rg, dim3(kThreads), 0, stream, dk_out, dk, n4, s.S,
                       s.Hkl * D, ck.n, ck.rows);
  }

  const int qtiles = (s.S + kDQM - 1) / kDQM;
  const int heads_total = s.b * s.Hl;
  hipLaunchKernelGGL(bwd_dq_kernel<D>, dim3((unsigned)(qtiles * heads_total)), dim3(kThreads),
                     0, stream, qp, kp, vp, dop, lse, Dbuf, dq, s.S, s.Hl, s.Hkl, n_rep,
                     heads_total, qtiles, c, s.scale);
  return hipGetLastError();
}

}  // namespace

size_t attn_bwd_workspace_bytes(const AttnShape &s) {
  const BwdChunks ck = bwd_chunks(s);
  size_t floats = ck.part_offset_floats;
  if (ck.n > 1) floats += 2 * (size_t)ck.n * s.b * s.Hkl * s.S * s.d;
  return floats * sizeof(float);
}

hipError_t launch_attn_bwd(const void *q, const void *k, const void *v,
                           const void *o, const float *lse, const void *d_o,
                           float *dq, float *dk, float *dv, void *workspace,
                           const AttnShape &s, hipStream_t stream) {
  if ((long long)s.b * s.S == 0) return hipSuccess;
  float *Dbuf = static_cast<float *>(workspace);
  if (s.d == 128)
    return launch_bwd_d<128>(q, k, v, o, lse, d_o, dq, dk, dv, Dbuf, s, stream);
  return launch_bwd_d<64>(q, k, v, o, lse, d_o, dq, dk, dv, Dbuf, s, stream);
}

}  // namespace basp
