// basp_attn_fwd.hip -- causal GQA attention forward for the rank's heads.
//
// Computes the scaled dot-product attention of Sec. II-A of the paper over
// the full sequence, masked causally (key j visible to query i iff j <= i),
// for each local query head h with local kv head h / n_rep:
//   O_i = sum_j softmax_j(scale * q_i . k_j) v_j,   LSE_i = log sum_j exp(.)
// The S x S score matrix is never stored: keys are visited in tiles with a
// running row maximum and row sum (online softmax), the standard
// re-association that changes only rounding.
//
// gfx950 mapping
//   * workgroup = 4 waves = 128 query rows of one (sequence, head); wave w
//     owns rows q0 + 32w .. +31, one row per lane pair (l, l+32).
//   * scores are formed transposed, S^T = K Q^T, with
//     v_mfma_f32_32x32x16_bf16: K (A operand) from LDS, Q (B operand) kept
//     in registers for the whole loop.  The 32x32 accumulator then gives each
//     lane one query row and 16 keys, so the softmax statistics are lane-local
//     up to one exchange with the partner lane l^32.
//   * O^T = V^T P^T: P goes from the score accumulator straight into the B
//     operand (bf16, round to nearest even); V^T (A operand) is read from a
//     transposed LDS copy whose key order inside each 16-block matches the
//     accumulator's row order (see mfma_pos16).
//   * K/V tiles of 64 keys are double-buffered in LDS and prefetched into
//     registers one tile ahead; tiles past a wave's last row are skipped and
//     only tiles crossing the diagonal are masked.
//   * the grid is one-dimensional, heaviest query tiles first (they visit the
//     most key tiles), heads fastest so that the heads sharing a kv head run
//     side by side.
#include <math.h>

#include "basp_device.hpp"
#include "basp_internal.hpp"

namespace basp {
namespace {

constexpr int kThreads = 256;
constexpr int kBM = 128;  // query rows per workgroup
constexpr int kBN = 64;   // keys per tile

template <int D>
struct FwdCfg {
  static constexpr int KS = D + 8;     // K tile row stride (elements), 16B-padded
  static constexpr int VS = kBN + 8;   // V^T row stride
  static constexpr int K_ELEMS = kBN * KS;
  static constexpr int V_ELEMS = D * VS;
  static constexpr int STAGE = K_ELEMS + V_ELEMS;
  static constexpr int NS = D / 16;    // 16-deep steps over the head dim
  static constexpr int NE = D / 32;    // 32-wide head-dim subtiles of O
  static constexpr int K_CHUNKS = kBN * D / 8 / kThreads;        // 16B chunks / thread
  static constexpr int V_UNITS = (kBN / 8) * (D / 2) / kThreads;  // 8 rows x 2 cols units
  static_assert(K_CHUNKS >= 1 && V_UNITS >= 1, "tile too small for the block");
};

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ k,
    const uint16_t *__restrict__ v, uint16_t *__restrict__ o,
    float *__restrict__ lse, int S, int Hl, int Hkl, int n_rep, int heads_total,
    int qtiles, float c /* scale * log2(e) */) {
  using C = FwdCfg<D>;
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * C::STAGE];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, hh = lane >> 5;

  const int L = blockIdx.x;
  const int qt = qtiles - 1 - L / heads_total;
  const int hb = L % heads_total;
  const int beta = hb / Hl, h = hb % Hl, kvh = h / n_rep;
  const int q0 = qt * kBM;
  const int wrow0 = q0 + 32 * w;
  const int row = wrow0 + l32;

  const size_t qstride = (size_t)Hl * D, kvstride = (size_t)Hkl * D;
  const uint16_t *qb = q + ((size_t)beta * S * Hl + h) * D;
  const uint16_t *kb = k + ((size_t)beta * S * Hkl + kvh) * D;
  const uint16_t *vb = v + ((size_t)beta * S * Hkl + kvh) * D;

  // Q fragments (B operand of S^T = K Q^T): row `row`, e = 16s + 8hh .. +7.
  bf16x8 qf[C::NS];
  {
    const u32x4 zero = {0u, 0u, 0u, 0u};
    const u32x4 *src = reinterpret_cast<const u32x4 *>(qb + (size_t)row * qstride);
#pragma unroll
    for (int s = 0; s < C::NS; ++s) qf[s] = as_bf16x8(row < S ? src[2 * s + hh] : zero);
  }

  const int kv_end = min(S, q0 + kBM);
  const int nt = (kv_end + kBN - 1) / kBN;

  u32x4 kreg[C::K_CHUNKS];
  uint32_t vreg[C::V_UNITS][8];

  auto load_tile = [&](int t) {
    const int j0 = t * kBN;
#pragma unroll
    for (int r = 0; r < C::K_CHUNKS; ++r) {
      const int cidx = tid + r * kThreads;
      const int jr = cidx / (D / 8), c8 = cidx % (D / 8);
      const int j = j0 + jr;
      const u32x4 zero = {0u, 0u, 0u, 0u};
      kreg[r] = j < S ? reinterpret_cast<const u32x4 *>(kb + (size_t)j * kvstride)[c8] : zero;
    }
#pragma unroll
    for (int u = 0; u < C::V_UNITS; ++u) {
      const int uidx = tid + u * kThreads;
      const int ep = uidx % (D / 2), jg = uidx / (D / 2);
      const int blk = jg >> 1, half = jg & 1;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int j = j0 + blk * 16 + half * 4 + (r & 3) + (r >> 2) * 8;
        vreg[u][r] = j < S ? reinterpret_cast<const uint32_t *>(vb + (size_t)j * kvstride)[ep] : 0u;
      }
    }
  };

  auto store_tile = [&](int buf) {
    uint16_t *Ks = smem + buf * C::STAGE;
    uint16_t *Vt = Ks + C::K_ELEMS;
#pragma unroll
    for (int r = 0; r < C::K_CHUNKS; ++r) {
      const int cidx = tid + r * kThreads;
      const int jr = cidx / (D / 8), c8 = cidx % (D / 8);
      *reinterpret_cast<u32x4 *>(Ks + jr * C::KS + c8 * 8) = kreg[r];
    }
#pragma unroll
    for (int u = 0; u < C::V_UNITS; ++u) {
      const int uidx = tid + u * kThreads;
      const int ep = uidx % (D / 2), jg = uidx / (D / 2);
      const int pos = (jg >> 1) * 16 + (jg & 1) * 8;
      const uint32_t *x = vreg[u];
      u32x4 lo = {lo_halves(x[0], x[1]), lo_halves(x[2], x[3]), lo_halves(x[4], x[5]),
                  lo_halves(x[6], x[7])};
      u32x4 hi = {hi_halves(x[0], x[1]), hi_halves(x[2], x[3]), hi_halves(x[4], x[5]),
                  hi_halves(x[6], x[7])};
      *reinterpret_cast<u32x4 *>(Vt + (2 * ep) * C::VS + pos) = lo;
      *reinterpret_cast<u32x4 *>(Vt + (2 * ep + 1) * C::VS + pos) = hi;
    }
  };

  f32x16 oacc[C::NE];
#pragma unroll
  for (int n = 0; n < C::NE; ++n)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[n][r] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  load_tile(0);
  store_tile(0);
  __syncthreads();

  for (int t = 0; t < nt; ++t) {
    if (t + 1 < nt) load_tile(t + 1);
    const int j0 = t * kBN;
    if (j0 <= wrow0 + 31) {  // wave-uniform: tile has keys visible to this wave
      const uint16_t *Ks = smem + (t & 1) * C::STAGE;
      const uint16_t *Vt = Ks + C::K_ELEMS;

      f32x16 sacc[2];
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) sacc[m][r] = 0.f;
#pragma unroll
      for (int s = 0; s < C::NS; ++s)
#pragma unroll
        for (int m = 0; m < 2; ++m) {
          const bf16x8 a =
              *reinterpret_cast<const bf16x8 *>(Ks + (32 * m + l32) * C::KS + 16 * s + 8 * hh);
          sacc[m] = mfma32x32x16(a, qf[s], sacc[m]);
        }

      // sacc[m][r] = S^T[key j0 + 32m + 8(r/4) + 4hh + r%4][query row]
      if (j0 + kBN - 1 > wrow0) {
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
      mx = fmaxf(mx, swap_halves(mx));
      const float m_new = fmaxf(m_run, mx * c);
      const float alpha = fast_exp2(m_run - m_new);
      m_run = m_new;
      float psum = 0.f;
#pragma unroll
      for (int m = 0; m < 2; ++m)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = fast_exp2(fmaf(sacc[m][r], c, -m_new));
          sacc[m][r] = p;
          psum += p;
        }
      l_run = l_run * alpha + psum;
#pragma unroll
      for (int n = 0; n < C::NE; ++n)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[n][r] *= alpha;

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
          const bf16x8 a =
              *reinterpret_cast<const bf16x8 *>(Vt + (32 * n + l32) * C::VS + 16 * s2 + 8 * hh);
          oacc[n] = mfma32x32x16(a, pf[s2], oacc[n]);
        }
    }
    if (t + 1 < nt) store_tile((t + 1) & 1);
    __syncthreads();
  }

  // oacc[n][r] = O^T[e = 32n + 8(r/4) + 4hh + r%4][query row] (unnormalised)
  const float l_tot = l_run + swap_halves(l_run);
  if (row < S) {
    const float inv = 1.f / l_tot;
    uint16_t *ob = o + ((size_t)(beta * S + row) * Hl + h) * D;
#pragma unroll
    for (int n = 0; n < C::NE; ++n)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        u32x2 val = {pack_bf16x2(oacc[n][4 * g] * inv, oacc[n][4 * g + 1] * inv),
                     pack_bf16x2(oacc[n][4 * g + 2] * inv, oacc[n][4 * g + 3] * inv)};
        *reinterpret_cast<u32x2 *>(ob + 32 * n + 8 * g + 4 * hh) = val;
      }
    if (hh == 0)
      lse[((size_t)beta * Hl + h) * S + row] = (m_run + fast_log2(l_tot)) * 0.69314718055994531f;
  }
}

}  // namespace

hipError_t launch_attn_fwd(const void *q, const void *k, const void *v, void *o,
                           float *lse, const AttnShape &s, hipStream_t stream) {
  const int qtiles = (s.S + kBM - 1) / kBM;
  const int heads_total = s.b * s.Hl;
  const long long blocks = (long long)qtiles * heads_total;
  if (blocks == 0) return hipSuccess;
  const float c = s.scale * 1.4426950408889634f;
  const int n_rep = s.Hl / s.Hkl;
  auto *qp = static_cast<const uint16_t *>(q);
  auto *kp = static_cast<const uint16_t *>(k);
  auto *vp = static_cast<const uint16_t *>(v);
  auto *op = static_cast<uint16_t *>(o);
  if (s.d == 128)
    hipLaunchKernelGGL(attn_fwd_kernel<128>, dim3((unsigned)blocks), dim3(kThreads), 0, stream,
                       qp, kp, vp, op, lse, s.S, s.Hl, s.Hkl, n_rep, heads_total, qtiles, c);
  else
    hipLaunchKernelGGL(attn_fwd_kernel<64>, dim3((unsigned)blocks), dim3(kThreads), 0, stream,
                       qp, kp, vp, op, lse, s.S, s.Hl, s.Hkl, n_rep, heads_total, qtiles, c);
  return hipGetLastError();
}

}  // namespace basp
