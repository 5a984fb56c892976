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
// Three kernels, all deterministic (no atomics):
//   bwd_pre   D for every (sequence, head, row)
//   bwd_dkdv  key-stationary: a workgroup owns 128 keys of one kv head and
//             sweeps every query row at or after them, for all query heads
//             of the GQA group, accumulating dK and dV in registers
//   bwd_dq    query-stationary: like the forward, a workgroup owns 128 rows
//             of one query head and sweeps the keys up to the diagonal
// On gfx950 both main kernels use v_mfma_f32_32x32x16_bf16 with fp32
// accumulation.  Which operand order is used is chosen so that every
// elementwise step (P, dS) happens in the accumulator layout and feeds the
// next product without a round trip through LDS; the operands that must be
// read along the sequence are kept in transposed LDS copies whose order
// inside each 16-block matches the accumulator (mfma_pos16).
#include <math.h>

#include "basp_device.hpp"
#include "basp_internal.hpp"

namespace basp {
namespace {

constexpr int kThreads = 256;
constexpr float kLog2e = 1.4426950408889634f;

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

// ---------------------------------------------------------------- bwd_dkdv
constexpr int kKN = 128;  // keys per workgroup (32 per wave)
constexpr int kQM = 64;   // query rows per step

template <int D>
struct DkdvCfg {
  static constexpr int RS = D + 8;    // row-major tile stride (elements)
  static constexpr int TS = kQM + 8;  // transposed tile stride
  static constexpr int ROW_ELEMS = kQM * RS;
  static constexpr int T_ELEMS = D * TS;
  // Q, dO row-major; Q^T, dO^T transposed; then 2 x kQM floats (LSE2, D).
  static constexpr int STAGE_BYTES = (2 * ROW_ELEMS + 2 * T_ELEMS) * 2 + 2 * kQM * 4;
  static constexpr int NS = D / 16;
  static constexpr int NE = D / 32;
  static constexpr int UNITS = (kQM / 8) * (D / 2) / kThreads;  // 8 rows x 2 cols per unit
  static_assert(UNITS >= 1, "tile too small");
};

template <int D>
__global__ __launch_bounds__(kThreads, 1) void bwd_dkdv_kernel(
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k,
    const uint16_t *__restrict__ v, const uint16_t *__restrict__ d_o,
    const float *__restrict__ lse, const float *__restrict__ Dbuf,
    float *__restrict__ dk, float *__restrict__ dv, int S, int Hl, int Hkl,
    int n_rep, int kvheads_total, float c /* scale*log2e */, float scale) {
  using C = DkdvCfg<D>;
  __shared__ __attribute__((aligned(16))) unsigned char smem[2 * C::STAGE_BYTES];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int L = blockIdx.x;
  const int kt = L / kvheads_total;  // heaviest (earliest keys) first
  const int hb = L % kvheads_total;
  const int beta = hb / Hkl, kvh = hb % Hkl;
  const int k0 = kt * kKN;
  const int wk0 = k0 + 32 * w;
  const int key = wk0 + l32;

  const size_t qstride = (size_t)Hl * D, kvstride = (size_t)Hkl * D;
  const uint16_t *kb = k + ((size_t)beta * S * Hkl + kvh) * D;
  const uint16_t *vb = v + ((size_t)beta * S * Hkl + kvh) * D;

  // K and V of this lane's key as B operands (B[e][j] = K[j][e]).
  bf16x8 kf[C::NS], vf[C::NS];
  {
    const u32x4 zero = {0u, 0u, 0u, 0u};
    const u32x4 *ks = reinterpret_cast<const u32x4 *>(kb + (size_t)key * kvstride);
    const u32x4 *vs = reinterpret_cast<const u32x4 *>(vb + (size_t)key * kvstride);
#pragma unroll
    for (int s = 0; s < C::NS; ++s) {
      kf[s] = as_bf16x8(key < S ? ks[2 * s + hh] : zero);
      vf[s] = as_bf16x8(key < S ? vs[2 * s + hh] : zero);
    }
  }

  f32x16 dkacc[C::NE], dvacc[C::NE];
#pragma unroll
  for (int n = 0; n < C::NE; ++n)
#pragma unroll
    for (int r = 0; r < 16; ++r) dkacc[n][r] = dvacc[n][r] = 0.f;

  const int qt0 = k0 / kQM;
  const int qtn = (S + kQM - 1) / kQM;
  const int steps_per_head = qtn - qt0;
  const int nsteps = steps_per_head * n_rep;

  uint32_t qreg[C::UNITS][8], doreg[C::UNITS][8];
  float aux = 0.f;  // LSE2 (tid < 64) or D (64 <= tid < 128) of one row

  auto step_coords = [&](int st, int &h, int &i0) {
    const int hr = st / steps_per_head;
    h = kvh * n_rep + hr;
    i0 = (qt0 + (st - hr * steps_per_head)) * kQM;
  };

  auto load_step = [&](int st) {
    int h, i0;
    step_coords(st, h, i0);
    const uint16_t *qb = q + ((size_t)beta * S * Hl + h) * D;
    const uint16_t *db = d_o + ((size_t)beta * S * Hl + h) * D;
#pragma unroll
    for (int u = 0; u < C::UNITS; ++u) {
      const int uidx = tid + u * kThreads;
      const int ep = uidx % (D / 2), ig = uidx / (D / 2);
      const int blk = ig >> 1, half = ig & 1;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int i = i0 + blk * 16 + half * 4 + (r & 3) + (r >> 2) * 8;
        const bool ok = i < S;
        qreg[u][r] = ok ? reinterpret_cast<const uint32_t *>(qb + (size_t)i * qstride)[ep] : 0u;
        doreg[u][r] = ok ? reinterpret_cast<const uint32_t *>(db + (size_t)i * qstride)[ep] : 0u;
      }
    }
    if (tid < 2 * kQM) {
      const int i = i0 + (tid & (kQM - 1));
      const size_t idx = ((size_t)beta * Hl + h) * S + i;
      if (tid < kQM)
        aux = i < S ? lse[idx] * kLog2e : INFINITY;
      else
        aux = i < S ? Dbuf[idx] : 0.f;
    }
  };

  auto store_step = [&](int buf) {
    unsigned char *base = smem + buf * C::STAGE_BYTES;
    uint16_t *Qs = reinterpret_cast<uint16_t *>(base);
    uint16_t *dOs = Qs + C::ROW_ELEMS;
    uint16_t *Qt = dOs + C::ROW_ELEMS;
    uint16_t *dOt = Qt + C::T_ELEMS;
    float *aux_s = reinterpret_cast<float *>(dOt + C::T_ELEMS);
#pragma unroll
    for (int u = 0; u < C::UNITS; ++u) {
      const int uidx = tid + u * kThreads;
      const int ep = uidx % (D / 2), ig = uidx / (D / 2);
      const int blk = ig >> 1, half = ig & 1;
      const int pos = blk * 16 + half * 8;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int il = blk * 16 + half * 4 + (r & 3) + (r >> 2) * 8;
        *reinterpret_cast<uint32_t *>(Qs + il * C::RS + 2 * ep) = qreg[u][r];
        *reinterpret_cast<uint32_t *>(dOs + il * C::RS + 2 * ep) = doreg[u][r];
      }
      const uint32_t *x = qreg[u];
      const uint32_t *y = doreg[u];
      u32x4 qlo = {lo_halves(x[0], x[1]), lo_halves(x[2], x[3]), lo_halves(x[4], x[5]),
                   lo_halves(x[6], x[7])};
      u32x4 qhi = {hi_halves(x[0], x[1]), hi_halves(x[2], x[3]), hi_halves(x[4], x[5]),
                   hi_halves(x[6], x[7])};
      u32x4 dlo = {lo_halves(y[0], y[1]), lo_halves(y[2], y[3]), lo_halves(y[4], y[5]),
                   lo_halves(y[6], y[7])};
      u32x4 dhi = {hi_halves(y[0], y[1]), hi_halves(y[2], y[3]), hi_halves(y[4], y[5]),
                   hi_halves(y[6], y[7])};
      *reinterpret_cast<u32x4 *>(Qt + (2 * ep) * C::TS + pos) = qlo;
      *reinterpret_cast<u32x4 *>(Qt + (2 * ep + 1) * C::TS + pos) = qhi;
      *reinterpret_cast<u32x4 *>(dOt + (2 * ep) * C::TS + pos) = dlo;
      *reinterpret_cast<u32x4 *>(dOt + (2 * ep + 1) * C::TS + pos) = dhi;
    }
    if (tid < 2 * kQM) aux_s[tid] = aux;
  };

  if (nsteps > 0) {
    load_step(0);
    store_step(0);
  }
  __syncthreads();

  for (int st = 0; st < nsteps; ++st) {
    if (st + 1 < nsteps) load_step(st + 1);
    int h_unused, i0;
    step_coords(st, h_unused, i0);
    if (i0 + kQM - 1 >= wk0) {  // wave-uniform: some row of the step sees a key of this wave
      const unsigned char *base = smem + (st & 1) * C::STAGE_BYTES;
      const uint16_t *Qs = reinterpret_cast<const uint16_t *>(base);
      const uint16_t *dOs = Qs + C::ROW_ELEMS;
      const uint16_t *Qt = dOs + C::ROW_ELEMS;
      const uint16_t *dOt = Qt + C::T_ELEMS;
      const float *lse_s = reinterpret_cast<const float *>(dOt + C::T_ELEMS);
      const float *D_s = lse_s + kQM;

      // S = Q K^T and dP = dO V^T: M = query rows (2 x 32), N = the wave's keys.
      f32x16 sacc[2], pacc[2];
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[m][r] = pacc[m][r] = 0.f;
#pragma unroll
      for (int s = 0; s < C::NS; ++s)
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          const bf16x8 aq =
              *reinterpret_cast<const bf16x8 *>(Qs + (32 * m + l32) * C::RS + 16 * s + 8 * hh);
          const bf16x8 ad =
              *reinterpret_cast<const bf16x8 *>(dOs + (32 * m + l32) * C::RS + 16 * s + 8 * hh);
          sacc[m] = mfma32x32x16(aq, kf[s], sacc[m]);
          pacc[m] = mfma32x32x16(ad, vf[s], pacc[m]);
        }
      // acc[m][r] holds row i0 + 32m + 8(r/4) + 4hh + r%4, key `key`.
      const bool diag = i0 < wk0 + 31;
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int il = 32 * m + 8 * g + 4 * hh;
          const f32x4 l4 = *reinterpret_cast<const f32x4 *>(lse_s + il);
          const f32x4 d4 = *reinterpret_cast<const f32x4 *>(D_s + il);
#pragma unroll
          for (int x = 0; x < 4; ++x) {
            const int r = 4 * g + x;
            float p = fast_exp2(fmaf(sacc[m][r], c, -l4[x]));
            if (diag && key > i0 + il + x) p = 0.f;
            sacc[m][r] = p;
            pacc[m][r] = p * (pacc[m][r] - d4[x]);
          }
        }
      // P and dS as B operands along the query rows: step s covers rows
      // 16s .. 16s+15 of the 64, slot t <-> accumulator register (s&1)*8 + t.
      bf16x8 pb[kQM / 16], sb[kQM / 16];
#pragma unroll
      for (int s2 = 0; s2 < kQM / 16; ++s2) {
        const int m = s2 >> 1, b8 = (s2 & 1) * 8;
        u32x4 tp = {pack_bf16x2(sacc[m][b8 + 0], sacc[m][b8 + 1]),
                    pack_bf16x2(sacc[m][b8 + 2], sacc[m][b8 + 3]),
                    pack_bf16x2(sacc[m][b8 + 4], sacc[m][b8 + 5]),
                    pack_bf16x2(sacc[m][b8 + 6], sacc[m][b8 + 7])};
        u32x4 ts = {pack_bf16x2(pacc[m][b8 + 0], pacc[m][b8 + 1]),
                    pack_bf16x2(pacc[m][b8 + 2], pacc[m][b8 + 3]),
                    pack_bf16x2(pacc[m][b8 + 4], pacc[m][b8 + 5]),
                    pack_bf16x2(pacc[m][b8 + 6], pacc[m][b8 + 7])};
        pb[s2] = as_bf16x8(tp);
        sb[s2] = as_bf16x8(ts);
      }
      // dV^T += dO^T P,  dK^T += Q^T dS:  M = head dim, N = keys, K = rows.
#pragma unroll
      for (int n = 0; n < C::NE; ++n)
#pragma unroll
        for (int s2 = 0; s2 < kQM / 16; ++s2) {
          const bf16x8 ad =
              *reinterpret_cast<const bf16x8 *>(dOt + (32 * n + l32) * C::TS + 16 * s2 + 8 * hh);
          const bf16x8 aq =
              *reinterpret_cast<const bf16x8 *>(Qt + (32 * n + l32) * C::TS + 16 * s2 + 8 * hh);
          dvacc[n] = mfma32x32x16(ad, pb[s2], dvacc[n]);
          dkacc[n] = mfma32x32x16(aq, sb[s2], dkacc[n]);
        }
    }
    if (st + 1 < nsteps) store_step((st + 1) & 1);
    __syncthreads();
  }

  // dkacc[n][r] = dK^T[e = 32n + 8(r/4) + 4hh + r%4][key]
  if (key < S) {
    float *dkr = dk + ((size_t)(beta * S + key) * Hkl + kvh) * D;
    float *dvr = dv + ((size_t)(beta * S + key) * Hkl + kvh) * D;
#pragma unroll
    for (int n = 0; n < C::NE; ++n)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 a = {dkacc[n][4 * g] * scale, dkacc[n][4 * g + 1] * scale,
                   dkacc[n][4 * g + 2] * scale, dkacc[n][4 * g + 3] * scale};
        f32x4 b = {dvacc[n][4 * g], dvacc[n][4 * g + 1], dvacc[n][4 * g + 2],
                   dvacc[n][4 * g + 3]};
        *reinterpret_cast<f32x4 *>(dkr + 32 * n + 8 * g + 4 * hh) = a;
        *reinterpret_cast<f32x4 *>(dvr + 32 * n + 8 * g + 4 * hh) = b;
      }
  }
}

// ---------------------------------------------------------------- bwd_dq
constexpr int kDQM = 128;  // query rows per workgroup (32 per wave)
constexpr int kDQN = 64;   // keys per tile

template <int D>
struct DqCfg {
  static constexpr int RS = D + 8;     // K, V row-major stride
  static constexpr int TS = kDQN + 8;  // K^T stride
  static constexpr int ROW_ELEMS = kDQN * RS;
  static constexpr int T_ELEMS = D * TS;
  static constexpr int STAGE = 2 * ROW_ELEMS + T_ELEMS;
  static constexpr int NS = D / 16;
  static constexpr int NE = D / 32;
  static constexpr int CHUNKS = kDQN * D / 8 / kThreads;
  static constexpr int UNITS = (kDQN / 8) * (D / 2) / kThreads;
  static_assert(CHUNKS >= 1 && UNITS >= 1, "tile too small");
};

template <int D>
__global__ __launch_bounds__(kThreads, 1) void bwd_dq_kernel(
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k,
    const uint16_t *__restrict__ v, const uint16_t *__restrict__ d_o,
    const float *__restrict__ lse, const float *__restrict__ Dbuf,
    float *__restrict__ dq, int S, int Hl, int Hkl, int n_rep, int heads_total,
    int qtiles, float c, float scale) {
  using C = DqCfg<D>;
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * C::STAGE];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;
  const int L = blockIdx.x;
  const int qt = qtiles - 1 - L / heads_total;
  const int hb = L % heads_total;
  const int beta = hb / Hl, h = hb % Hl, kvh = h / n_rep;
  const int q0 = qt * kDQM;
  const int wrow0 = q0 + 32 * w;
  const int row = wrow0 + l32;

  const size_t qstride = (size_t)Hl * D, kvstride = (size_t)Hkl * D;
  const uint16_t *qb = q + ((size_t)beta * S * Hl + h) * D;
  const uint16_t *db = d_o + ((size_t)beta * S * Hl + h) * D;
  const uint16_t *kb = k + ((size_t)beta * S * Hkl + kvh) * D;
  const uint16_t *vb = v + ((size_t)beta * S * Hkl + kvh) * D;

  bf16x8 qf[C::NS], df[C::NS];
  {
    const u32x4 zero = {0u, 0u, 0u, 0u};
    const u32x4 *qs = reinterpret_cast<const u32x4 *>(qb + (size_t)row * qstride);
    const u32x4 *ds = reinterpret_cast<const u32x4 *>(db + (size_t)row * qstride);
#pragma unroll
    for (int s = 0; s < C::NS; ++s) {
      qf[s] = as_bf16x8(row < S ? qs[2 * s + hh] : zero);
      df[s] = as_bf16x8(row < S ? ds[2 * s + hh] : zero);
    }
  }
  const size_t lidx = ((size_t)beta * Hl + h) * S + row;
  const float lse2 = row < S ? lse[lidx] * kLog2e : INFINITY;
  const float Drow = row < S ? Dbuf[lidx] : 0.f;

  const int kv_end = min(S, q0 + kDQM);
  const int nt = (kv_end + kDQN - 1) / kDQN;

  u32x4 kreg[C::CHUNKS], vreg[C::CHUNKS];
  uint32_t ktreg[C::UNITS][8];

  auto load_tile = [&](int t) {
    const int j0 = t * kDQN;
    const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int r = 0; r < C::CHUNKS; ++r) {
      const int cidx = tid + r * kThreads;
      const int jr = cidx / (D / 8), c8 = cidx % (D / 8);
      const int j = j0 + jr;
      kreg[r] = j < S ? reinterpret_cast<const u32x4 *>(kb + (size_t)j * kvstride)[c8] : zero;
      vreg[r] = j < S ? reinterpret_cast<const u32x4 *>(vb + (size_t)j * kvstride)[c8] : zero;
    }
#pragma unroll
    for (int u = 0; u < C::UNITS; ++u) {
      const int uidx = tid + u * kThreads;
      const int ep = uidx % (D / 2), jg = uidx / (D / 2);
      const int blk = jg >> 1, half = jg & 1;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int j = j0 + blk * 16 + half * 4 + (r & 3) + (r >> 2) * 8;
        ktreg[u][r] = j < S ? reinterpret_cast<const uint32_t *>(kb + (size_t)j * kvstride)[ep] : 0u;
      }
    }
  };

  auto store_tile = [&](int buf) {
    uint16_t *Ks = smem + buf * C::STAGE;
    uint16_t *Vs = Ks + C::ROW_ELEMS;
    uint16_t *Kt = Vs + C::ROW_ELEMS;
#pragma unroll
    for (int r = 0; r < C::CHUNKS; ++r) {
      const int cidx = tid + r * kThreads;
      const int jr = cidx / (D / 8), c8 = cidx % (D / 8);
      *reinterpret_cast<u32x4 *>(Ks + jr * C::RS + c8 * 8) = kreg[r];
      *reinterpret_cast<u32x4 *>(Vs + jr * C::RS + c8 * 8) = vreg[r];
    }
#pragma unroll
    for (int u = 0; u < C::UNITS; ++u) {
      const int uidx = tid + u * kThreads;
      const int ep = uidx % (D / 2), jg = uidx / (D / 2);
      const int pos = (jg >> 1) * 16 + (jg & 1) * 8;
      const uint32_t *x = ktreg[u];
      u32x4 lo = {lo_halves(x[0], x[1]), lo_halves(x[2], x[3]), lo_halves(x[4], x[5]),
                  lo_halves(x[6], x[7])};
      u32x4 hi = {hi_halves(x[0], x[1]), hi_halves(x[2], x[3]), hi_halves(x[4], x[5]),
                  hi_halves(x[6], x[7])};
      *reinterpret_cast<u32x4 *>(Kt + (2 * ep) * C::TS + pos) = lo;
      *reinterpret_cast<u32x4 *>(Kt + (2 * ep + 1) * C::TS + pos) = hi;
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
      const uint16_t *Ks = smem + (t & 1) * C::STAGE;
      const uint16_t *Vs = Ks + C::ROW_ELEMS;
      const uint16_t *Kt = Vs + C::ROW_ELEMS;
      // S^T = K Q^T and dP^T = V dO^T: M = keys (2 x 32), N = this wave's rows.
      f32x16 sacc[2], pacc[2];
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[m][r] = pacc[m][r] = 0.f;
#pragma unroll
      for (int s = 0; s < C::NS; ++s)
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          const bf16x8 ak =
              *reinterpret_cast<const bf16x8 *>(Ks + (32 * m + l32) * C::RS + 16 * s + 8 * hh);
          const bf16x8 av =
              *reinterpret_cast<const bf16x8 *>(Vs + (32 * m + l32) * C::RS + 16 * s + 8 * hh);
          sacc[m] = mfma32x32x16(ak, qf[s], sacc[m]);
          pacc[m] = mfma32x32x16(av, df[s], pacc[m]);
        }
      const bool diag = j0 + kDQN - 1 > wrow0;
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j = j0 + 32 * m + 8 * (r >> 2) + 4 * hh + (r & 3);
          float p = fast_exp2(fmaf(sacc[m][r], c, -lse2));
          if (diag && j > row) p = 0.f;
          pacc[m][r] = p * (pacc[m][r] - Drow);
        }
      bf16x8 sb[kDQN / 16];
#pragma unroll
      for (int s2 = 0; s2 < kDQN / 16; ++s2) {
        const int m = s2 >> 1, b8 = (s2 & 1) * 8;
        u32x4 ts = {pack_bf16x2(pacc[m][b8 + 0], pacc[m][b8 + 1]),
                    pack_bf16x2(pacc[m][b8 + 2], pacc[m][b8 + 3]),
                    pack_bf16x2(pacc[m][b8 + 4], pacc[m][b8 + 5]),
                    pack_bf16x2(pacc[m][b8 + 6], pacc[m][b8 + 7])};
        sb[s2] = as_bf16x8(ts);
      }
      // dQ^T += K^T dS^T: M = head dim, N = rows, K = keys.
#pragma unroll
      for (int n = 0; n < C::NE; ++n)
#pragma unroll
        for (int s2 = 0; s2 < kDQN / 16; ++s2) {
          const bf16x8 a =
              *reinterpret_cast<const bf16x8 *>(Kt + (32 * n + l32) * C::TS + 16 * s2 + 8 * hh);
          qacc[n] = mfma32x32x16(a, sb[s2], qacc[n]);
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
  hipLaunchKernelGGL(bwd_dkdv_kernel<D>, dim3((unsigned)(ktiles * kvheads_total)),
                     dim3(kThreads), 0, stream, qp, kp, vp, dop, lse, Dbuf, dk, dv, s.S,
                     s.Hl, s.Hkl, n_rep, kvheads_total, c, s.scale);

  const int qtiles = (s.S + kDQM - 1) / kDQM;
  const int heads_total = s.b * s.Hl;
  hipLaunchKernelGGL(bwd_dq_kernel<D>, dim3((unsigned)(qtiles * heads_total)), dim3(kThreads),
                     0, stream, qp, kp, vp, dop, lse, Dbuf, dq, s.S, s.Hl, s.Hkl, n_rep,
                     heads_total, qtiles, c, s.scale);
  return hipGetLastError();
}

}  // namespace

size_t attn_bwd_workspace_bytes(const AttnShape &s) {
  const size_t n = (size_t)s.b * s.Hl * s.S * sizeof(float);
  return (n + 255) & ~(size_t)255;
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
