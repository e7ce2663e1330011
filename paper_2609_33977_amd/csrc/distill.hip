// Self-distillation loss of the student against the dense teacher (Sec. 2.4,
// Eq. 4) through the frozen LM head W [V, d]:
//
//   z_T = H_T W^T,  z_S = H_S W^T                       (teacher, student logits)
//   L   = -(1/N) sum_{valid t} sum_v p_T(t, v) log p_S(t, v)
//       =  (1/N) sum_{valid t} ( lse_S(t) - sum_v p_T(t, v) z_S(t, v) )
//   dL/dz_S(t, v) = (p_S(t, v) - p_T(t, v)) / N,   dH_S = dz_S W
//
// Forward: one GEMM launch computes both passes' logits for a tile of 256
// vocabulary rows x 128 tokens (the W tile feeds the teacher and the student
// halves of the token tile), stores them in fp32, and reduces the tile to five
// statistics per token: the teacher's max and sum of exp, the student's, and
// the teacher-weighted sum of the student logits.  A per-token pass merges the
// vocabulary tiles in fixed order (log-sum-exp of both passes, the per-token
// cross-entropy) and one block sums the valid tokens.
// Backward: an elementwise pass forms dz_S in bf16 from the stored logits,
// and a second GEMM multiplies it by W.  Storing the fp32 logits (8 bytes per
// token and vocabulary entry) costs one write and one read of HBM instead of
// recomputing both passes' logits in the backward, which is the cheaper side
// on a GPU with this much memory and bandwidth.
#include "gm_gemm.h"
#include "gm_launch.h"

#include <math.h>

namespace gm {

constexpr int kLmWaves = 8;
constexpr int kLmTokens = 128;  // tokens of each pass per forward tile
constexpr int kLmStats = 5;     // m_T, s_T, m_S, s_S, c per token and vocabulary tile
// MFMA rows of a wave tile issued after each slice's barrier in the K-loop:
// four measured 1.6 % faster for the backward GEMM and 0.6 % slower for the
// forward one (whose epilogue dominates), so the forward keeps one.
constexpr int kLmFwdRowsAfter = 1, kLmBwdRowsAfter = 4;

// (m, s) <- merge of two (max, sum of exp(x - max)) summaries; an empty one has m = -inf, s = 0.
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float mx = fmaxf(m, m2);
  if (mx == -INFINITY) return;
  s = s * expf(m - mx) + s2 * expf(m2 - mx);
  m = mx;
}

// Teacher summary with the weighted student sum c = sum exp(z_T - m) z_S, which scales like s.
__device__ __forceinline__ void lse_merge_c(float& m, float& s, float& c, float m2, float s2, float c2) {
  const float mx = fmaxf(m, m2);
  if (mx == -INFINITY) return;
  const float a = expf(m - mx), b = expf(m2 - mx);
  s = s * a + s2 * b;
  c = c * a + c2 * b;
  m = mx;
}

// ---------------------------------------------------------------- forward GEMM

// Tile: 256 vocabulary rows (M, K-major W rows) x 256 columns (N): columns
// 0..127 are tokens t0..t0+127 of the teacher, 128..255 the same tokens of the
// student.  Waves 2 (M) x 4 (N): waves with wn < 2 hold teacher logits, the
// others the student logits of the same tokens and rows.  part holds the
// statistics as [N][tiles of V][kLmStats].
__global__ __launch_bounds__(64 * kLmWaves) void lmhead_fwd_kernel(const uint16_t* __restrict__ Ht,
                                                                  const uint16_t* __restrict__ Hs,
                                                                  const uint16_t* __restrict__ W, int N, int d,
                                                                  int V, float* __restrict__ zt,
                                                                  float* __restrict__ zs, float* __restrict__ part) {
  constexpr int NW = kLmWaves, WN = NW / 2;
  constexpr int BM = 256, BN = 2 * kLmTokens, MB = 8, NB = BN / WN / 16;
  constexpr int PER_STAGE = 32 / NW, CA = PER_STAGE / 2, STAGES = 4;
  __shared__ u32x4 smem[2 * STAGES * BM * 4];  // the A and B rings; afterwards the teacher logits
  __shared__ float s_half[2][kLmTokens][kLmStats];
  u32x4(*As)[BM * 4] = reinterpret_cast<u32x4(*)[BM * 4]>(smem);
  u32x4(*Bs)[BN * 4] = reinterpret_cast<u32x4(*)[BN * 4]>(smem + STAGES * BM * 4);

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int tiles_m = (V + BM - 1) / BM, tiles_n = (N + kLmTokens - 1) / kLmTokens;
  int tm, tn;
  tile_coords(gridDim.x, tiles_m, tiles_n, tm, tn);
  const int v0 = tm * BM, t0 = tn * kLmTokens;
  const int nst = d / kBK;

  // Copies: W rows v0 + row; B rows 0..127 (waves 0-3) from H_T, 128..255 (waves 4-7) from H_S.
  uint32_t offA[CA], offB[CA];
#pragma unroll
  for (int j = 0; j < CA; ++j) {
    int row, c;
    km_dma_target((wave * CA + j) * 64 + lane, row, c);
    offA[j] = group_voffset(uint32_t((v0 + row) * d + 8 * c) * 2u, j);
    offB[j] = group_voffset(uint32_t((t0 + (row & (kLmTokens - 1))) * d + 8 * c) * 2u, j);
  }
  const uint16_t* Hb = wave < NW / 2 ? Ht : Hs;
  const uint32_t bytesW = uint32_t(V) * uint32_t(d) * 2u;
  const uint32_t bytesH = uint32_t(N) * uint32_t(d) * 2u;
  i32x4_t rA, rB;
  auto prepare = [&](int st) {
    const bool live = st < nst;
    const int k0 = live ? st * kBK : 0;
    rA = make_rsrc_grouped(W + k0, live ? bytesW - 2u * uint32_t(k0) : 0u);
    rB = make_rsrc_grouped(Hb + k0, live ? bytesH - 2u * uint32_t(k0) : 0u);
  };
  const uint32_t ldsA = lds_addr(As), ldsB = lds_addr(Bs);
  auto issue = [&](int st, int p) {
    const int j = p % CA;
    const uint32_t dst = (st % STAGES) * (BM * 64) + wave * CA * 1024;
    if (p < CA)
      dma16_group(j, rA, offA[j], ldsA + dst);
    else
      dma16_group(j, rB, offB[j], ldsB + dst);
  };
  f32x4 acc[MB][NB];
  gemm_mainloop<MB, NB, true, true, 0, 0, PER_STAGE, STAGES, kLmFwdRowsAfter>(
      As, Bs, nst, wm * 128, wn * NB * 16, lane, acc, prepare, issue, [](int) {}, [](int, const u32x4(&)[NB]) {});

  // Lane (q = l >> 4, r = l & 15) holds, for every (mb, nb), rows v .. v + 3 of token column tl.
  const bool teacher = wn < WN / 2;
  const int q = lane >> 4, r = lane & 15;
  auto vrow = [&](int mb) { return v0 + wm * 128 + mb * 16 + 4 * q; };
  auto tcol = [&](int nb) { return (wn % (WN / 2)) * 64 + nb * 16 + r; };  // token within the tile

  // 1. Both passes' logits to HBM (fp32, [N, V]; V is a multiple of 4, so a
  //    row quad is entirely inside or outside the vocabulary).
  float* zout = teacher ? zt : zs;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int v = vrow(mb), t = t0 + tcol(nb);
      if (t < N && v < V) *reinterpret_cast<f32x4*>(zout + int64_t(t) * V + v) = acc[mb][nb];
    }

  // 2. The teacher waves hand their logits to the student waves holding the
  //    same rows and tokens (slot by wave row, column pair, fragment and lane).
  f32x4* zl = reinterpret_cast<f32x4*>(smem);
  auto slot = [&](int mb, int nb) { return (((wm * 2 + (wn % 2)) * MB + mb) * NB + nb) * 64 + lane; };
  __syncthreads();  // every wave has left the K-loop (its copies drained)
  if (teacher) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) zl[slot(mb, nb)] = acc[mb][nb];
  }
  __syncthreads();

  // 3. The student waves reduce each token over their 128 rows: per lane over
  //    32 rows, then over the four lane groups; the two wave rows meet in LDS.
  if (!teacher) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float mt = -INFINITY, ms = -INFINITY;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const f32x4 ztv = zl[slot(mb, nb)];
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (vrow(mb) + k < V) {
            mt = fmaxf(mt, ztv[k]);
            ms = fmaxf(ms, acc[mb][nb][k]);
          }
      }
      float st = 0.0f, ss = 0.0f, c = 0.0f;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const f32x4 ztv = zl[slot(mb, nb)];
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (vrow(mb) + k < V) {
            const float e = expf(ztv[k] - mt);
            st += e;
            c += e * acc[mb][nb][k];
            ss += expf(acc[mb][nb][k] - ms);
          }
      }
#pragma unroll
      for (int x = 16; x <= 32; x <<= 1) {
        const float mt2 = __shfl_xor(mt, x), st2 = __shfl_xor(st, x), c2 = __shfl_xor(c, x);
        const float ms2 = __shfl_xor(ms, x), ss2 = __shfl_xor(ss, x);
        lse_merge_c(mt, st, c, mt2, st2, c2);
        lse_merge(ms, ss, ms2, ss2);
      }
      if (q == 0) {
        float* h = s_half[wm][tcol(nb)];
        h[0] = mt;
        h[1] = st;
        h[2] = ms;
        h[3] = ss;
        h[4] = c;
      }
    }
  }
  __syncthreads();
  if (tid < kLmTokens && t0 + tid < N) {
    const float* a = s_half[0][tid];
    const float* b = s_half[1][tid];
    float mt = a[0], st = a[1], ms = a[2], ss = a[3], c = a[4];
    lse_merge_c(mt, st, c, b[0], b[1], b[4]);
    lse_merge(ms, ss, b[2], b[3]);
    float* p = part + (int64_t(t0 + tid) * tiles_m + tm) * kLmStats;
    p[0] = mt;
    p[1] = st;
    p[2] = ms;
    p[3] = ss;
    p[4] = c;
  }
}

// ---------------------------------------------------------------- per token

// One wave per token: lane l merges vocabulary tiles l, l + 64, ... in fp64,
// then the lanes combine in a fixed butterfly order.
__device__ __forceinline__ void merge_d(double& m, double& s, double m2, double s2) {
  const double mx = fmax(m, m2);
  if (mx == -INFINITY) return;
  s = s * exp(m - mx) + s2 * exp(m2 - mx);
  m = mx;
}

__device__ __forceinline__ void merge_dc(double& m, double& s, double& c, double m2, double s2, double c2) {
  const double mx = fmax(m, m2);
  if (mx == -INFINITY) return;
  const double a = exp(m - mx), b = exp(m2 - mx);
  s = s * a + s2 * b;
  c = c * a + c2 * b;
  m = mx;
}

__global__ __launch_bounds__(256) void distill_token_kernel(const float* __restrict__ part, int ntiles, int N,
                                                           float* __restrict__ lse_t, float* __restrict__ lse_s,
                                                           float* __restrict__ ce, float* __restrict__ ce_out) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= N) return;  // whole wave
  const float* p = part + int64_t(t) * ntiles * kLmStats;
  double mt = -INFINITY, st = 0.0, c = 0.0, ms = -INFINITY, ss = 0.0;
  for (int i = lane; i < ntiles; i += 64) {
    const float* q = p + i * kLmStats;
    merge_dc(mt, st, c, q[0], q[1], q[4]);
    merge_d(ms, ss, q[2], q[3]);
  }
#pragma unroll
  for (int x = 1; x < 64; x <<= 1) {
    const double mt2 = __shfl_xor(mt, x), st2 = __shfl_xor(st, x), c2 = __shfl_xor(c, x);
    const double ms2 = __shfl_xor(ms, x), ss2 = __shfl_xor(ss, x);
    merge_dc(mt, st, c, mt2, st2, c2);
    merge_d(ms, ss, ms2, ss2);
  }
  if (lane == 0) {
    const double ls = ms + log(ss);
    const double x = ls - c / st;
    lse_t[t] = float(mt + log(st));
    lse_s[t] = float(ls);
    ce[t] = float(x);
    if (ce_out) ce_out[t] = float(x);
  }
}

// One block: the number of valid tokens, the mean cross-entropy over them
// (fp64, fixed-order tree), and each token's gradient weight 1/N or 0.
__global__ __launch_bounds__(256) void distill_loss_kernel(const float* __restrict__ ce,
                                                          const uint8_t* __restrict__ valid, int N,
                                                          float* __restrict__ loss, float* __restrict__ wtok) {
  __shared__ double s_sum[256];
  __shared__ int s_cnt[256];
  const int tid = threadIdx.x;
  double a = 0.0;
  int n = 0;
  for (int t = tid; t < N; t += 256) {
    const bool ok = valid == nullptr || valid[t] != 0;
    if (ok) {
      a += double(ce[t]);
      ++n;
    }
  }
  s_sum[tid] = a;
  s_cnt[tid] = n;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if (tid < w) {
      s_sum[tid] += s_sum[tid + w];
      s_cnt[tid] += s_cnt[tid + w];
    }
    __syncthreads();
  }
  const int nv = s_cnt[0];
  const float inv = nv > 0 ? float(1.0 / double(nv)) : 0.0f;
  if (tid == 0) *loss = nv > 0 ? float(s_sum[0] / double(nv)) : 0.0f;
  for (int t = tid; t < N; t += 256) wtok[t] = (valid == nullptr || valid[t] != 0) ? inv : 0.0f;
}

// ---------------------------------------------------------------- backward

// dZ[t, v] = w_t (exp(z_S - lse_S) - exp(z_T - lse_T)) in bf16, rows padded
// with zeros to ldv (a multiple of 32) for the K-loop of the next GEMM.  One
// thread per 8 entries of a row.
__global__ __launch_bounds__(256) void distill_dz_kernel(const float* __restrict__ zt, const float* __restrict__ zs,
                                                        const float* __restrict__ lse_t,
                                                        const float* __restrict__ lse_s,
                                                        const float* __restrict__ wtok, int N, int V, int ldv,
                                                        uint16_t* __restrict__ dz) {
  const int per_row = ldv / 8;
  const int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (e >= int64_t(N) * per_row) return;
  const int t = int(e / per_row), v = int(e % per_row) * 8;
  u32x4 out = zero16();
  const float w = wtok[t];
  if (v < V && w != 0.0f) {
    const float ls = lse_s[t], lt = lse_t[t];
    const f32x4* ps = reinterpret_cast<const f32x4*>(zs + int64_t(t) * V + v);
    const f32x4* pt = reinterpret_cast<const f32x4*>(zt + int64_t(t) * V + v);
    float g[8];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const f32x4 a = ps[h], b = pt[h];
#pragma unroll
      for (int k = 0; k < 4; ++k) g[4 * h + k] = w * (expf(a[k] - ls) - expf(b[k] - lt));
    }
    out = u32x4{pack_bf16x2(g[0], g[1]), pack_bf16x2(g[2], g[3]), pack_bf16x2(g[4], g[5]), pack_bf16x2(g[6], g[7])};
  }
  st16(dz + int64_t(t) * ldv + v, out);
}

// dH[t, j] = sum_v dZ[t, v] W[v, j]: tile 256 (j) x 256 (t), K = v.  W is
// [V, d] with K as its row index (MN-major tile, transposing reads); dZ rows
// are K-contiguous (K-major tile).  Waves 2 (j) x 4 (t).
__global__ __launch_bounds__(64 * kLmWaves) void lmhead_bwd_kernel(const uint16_t* __restrict__ dz, int ldv,
                                                                  const uint16_t* __restrict__ W, int N, int d,
                                                                  int V, uint16_t* __restrict__ dH) {
  constexpr int NW = kLmWaves, WN = NW / 2;
  constexpr int BM = 256, BN = 256, MB = 8, NB = BN / WN / 16;
  constexpr int PER_STAGE = 32 / NW, CA = PER_STAGE / 2, STAGES = 4;
  __shared__ u32x4 As[STAGES][kBK * BM / 8];
  __shared__ u32x4 Bs[STAGES][BN * 4];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int tiles_m = (d + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  int tm, tn;
  tile_coords(gridDim.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int nst = ldv / kBK;

  uint32_t offA[CA], offB[CA];
#pragma unroll
  for (int j = 0; j < CA; ++j) {
    int row, c;
    mn_dma_target<BM>((wave * CA + j) * 64 + lane, row, c);
    offA[j] = group_voffset(m0 + 8 * c < d ? uint32_t(row * d + m0 + 8 * c) * 2u : kOOB, j);
    km_dma_target((wave * CA + j) * 64 + lane, row, c);
    offB[j] = group_voffset(uint32_t((n0 + row) * ldv + 8 * c) * 2u, j);
  }
  const uint32_t bytesW = uint32_t(V) * uint32_t(d) * 2u;
  const uint32_t bytesZ = uint32_t(N) * uint32_t(ldv) * 2u;
  i32x4_t rA, rB;
  auto prepare = [&](int st) {
    const bool live = st < nst;
    const int k0 = live ? st * kBK : 0;
    const uint32_t wskip = uint32_t(k0) * uint32_t(d) * 2u;
    rA = make_rsrc_grouped(W + int64_t(k0) * d, live && wskip < bytesW ? bytesW - wskip : 0u);
    rB = make_rsrc_grouped(dz + k0, live ? bytesZ - 2u * uint32_t(k0) : 0u);
  };
  const uint32_t ldsA = lds_addr(As), ldsB = lds_addr(Bs);
  auto issue = [&](int st, int p) {
    const int j = p % CA;
    const uint32_t dst = (st % STAGES) * (kBK * BM * 2) + wave * CA * 1024;
    if (p < CA)
      dma16_group(j, rA, offA[j], ldsA + dst);
    else
      dma16_group(j, rB, offB[j], ldsB + dst);
  };
  f32x4 acc[MB][NB];
  gemm_mainloop<MB, NB, false, true, BM, 0, PER_STAGE, STAGES, kLmBwdRowsAfter>(
      As, Bs, nst, wm * 128, wn * NB * 16, lane, acc, prepare, issue, [](int) {}, [](int, const u32x4(&)[NB]) {});
  store_tile_rows<BM, MB, NB, NW>(acc, reinterpret_cast<char*>(&As[0][0]), reinterpret_cast<char*>(&Bs[0][0]), wm, wn,
                                  tid, lane, dH, d, n0, N, m0, d);
}

// ---------------------------------------------------------------- launchers

int distill_vocab_tiles(int V) { return (V + 255) / 256; }

hipError_t launch_distill_fwd(const uint16_t* Ht, const uint16_t* Hs, const uint16_t* W, const uint8_t* valid, int N,
                              int d, int V, float* zt, float* zs, float* part, float* lse_t, float* lse_s, float* ce,
                              float* wtok, float* loss, float* ce_out, hipStream_t s) {
  const int tiles_m = distill_vocab_tiles(V), tiles_n = (N + kLmTokens - 1) / kLmTokens;
  hipLaunchKernelGGL(lmhead_fwd_kernel, dim3(unsigned(tiles_m * tiles_n)), dim3(64 * kLmWaves), 0, s, Ht, Hs, W, N, d,
                     V, zt, zs, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(distill_token_kernel, dim3(unsigned((N + 3) / 4)), dim3(256), 0, s, part, tiles_m, N, lse_t,
                     lse_s, ce, ce_out);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(distill_loss_kernel, dim3(1), dim3(256), 0, s, ce, valid, N, loss, wtok);
  return hipGetLastError();
}

hipError_t launch_distill_bwd(const uint16_t* W, int N, int d, int V, const float* zt, const float* zs,
                              const float* lse_t, const float* lse_s, const float* wtok, uint16_t* dz, int ldv,
                              uint16_t* dH, hipStream_t s) {
  const int64_t chunks = int64_t(N) * (ldv / 8);
  hipLaunchKernelGGL(distill_dz_kernel, dim3(unsigned((chunks + 255) / 256)), dim3(256), 0, s, zt, zs, lse_t, lse_s,
                     wtok, N, V, ldv, dz);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int tiles = ((d + 255) / 256) * ((N + 255) / 256);
  hipLaunchKernelGGL(lmhead_bwd_kernel, dim3(unsigned(tiles)), dim3(64 * kLmWaves), 0, s, dz, ldv, W, N, d, V, dH);
  return hipGetLastError();
}

}  // namespace gm
