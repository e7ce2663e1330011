// bf16 MFMA GEMMs of the group-masked linear layer on gfx950.
//
//   fwd   Y[t, o]  = sum_v mask[o, v] sum_{i in v} X[t, i] W[o, i]        (Eq. 1)
//   dX    dX[t, i] = sum_{o kept in group column v(i)} mask[o, v] dY[t, o] W[o, i]
//   dgate dgate[o, v] = sum_{i in v} W[o, i] sum_t dY[t, o] X[t, i]
//
// Common machinery: 256 x 256 output tiles (dX: 256 x min(g, 256)), K staged
// 64 at a time through double-buffered LDS tiles stored K-major with an XOR
// swizzle, eight waves per block, v_mfma_f32_16x16x32_bf16 with fp32
// accumulation, one block barrier per K stage.
//
// Operands that are stored with K strided in HBM (dY and X in dgate, the
// gathered rows of dY^T and W in dX) are transposed on their way into LDS:
// each staging thread loads an 8 x 8 bf16 block (eight 16-byte rows), swaps it
// in registers and writes eight K-contiguous 16-byte chunks.
//
// dgate's group reduction is fused into the epilogue: the fp32 tile of dY^T X
// is multiplied by W and summed over each group of g columns in registers and
// across lanes, so neither dY^T X nor any weight gradient reaches HBM.  The
// same kernel writes dY^T as a side output (from the blocks of the first
// column of tiles), which the dX GEMM reads to gather whole kept rows.
//
// dX runs one group column per tile: its K-loop walks only the kept rows of
// that column (the group-compacted column lists), so pruned groups cost
// nothing.  The forward skips every group column that no row of the tile
// keeps and never reads a pruned group's weights (zeros are staged instead).
#include "gm_device.h"
#include "gm_launch.h"

namespace gm {

constexpr int BK = 64;

// Blocks are handed to the eight XCDs round-robin; renumber them so that each
// XCD works on a contiguous range of tiles and shares operand panels in its L2.
__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
  const int per = nblocks / 8;
  if (per == 0 || bid >= per * 8) return bid;
  return (bid % 8) * per + bid / 8;
}

// One MFMA K stage of 64 for a wave tile of MB x NB 16x16 blocks.
template <int MB, int NB>
__device__ __forceinline__ void mma_stage(const u32x4* __restrict__ As, const u32x4* __restrict__ Bs, int arow0,
                                          int brow0, int lane, f32x4 (&acc)[MB][NB]) {
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const int kc = 4 * ks + (lane >> 4);
    u32x4 af[MB], bf[NB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) af[mb] = As[swz64(arow0 + mb * 16 + (lane & 15), kc)];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) bf[nb] = Bs[swz64(brow0 + nb * 16 + (lane & 15), kc)];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = mfma16x16x32(af[mb], bf[nb], acc[mb][nb]);
  }
}

template <int MB, int NB>
__device__ __forceinline__ void zero_acc(f32x4 (&acc)[MB][NB]) {
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// Write a K-contiguous transposed 8x8 block: LDS rows 8c .. 8c+7, k-chunk a.
__device__ __forceinline__ void store_transposed(u32x4* __restrict__ tile, int c, int a, const u32x4 (&v)[8],
                                                 u32x4 (&tr)[8]) {
  transpose8x8_b16(v, tr);
#pragma unroll
  for (int cc = 0; cc < 8; ++cc) tile[swz64(8 * c + cc, a)] = tr[cc];
}

// Store a wave's fp32 accumulator tile as bf16 rows of a row-major matrix.
template <int MB, int NB>
__device__ __forceinline__ void store_bf16_tile(const f32x4 (&acc)[MB][NB], uint16_t* __restrict__ out, int ld,
                                                int row0, int col0, int nrows, int ncols, int lane) {
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = row0 + mb * 16 + 4 * (lane >> 4) + j;
      if (r >= nrows) continue;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int c = col0 + nb * 16 + (lane & 15);
        if (c < ncols) out[int64_t(r) * ld + c] = uint16_t(f32_to_bf16_bits(acc[mb][nb][j]));
      }
    }
}

// ============================================================================ dgate

// Tile: 256 rows of W (o) x 256 columns (i); K = T.  Waves 2 (o) x 4 (i),
// wave tile 128 x 64.  For g = 512 a group spans two tiles: each adds its half
// to a zero-initialised dgate, and with exactly two addends onto zero the sum
// is the same whichever tile lands first.
template <int G>
__global__ __launch_bounds__(512) void dgate_kernel(const uint16_t* __restrict__ dY, const uint16_t* __restrict__ X,
                                                    const uint16_t* __restrict__ W, int T, int d_in, int d_out,
                                                    float* __restrict__ dgate, uint16_t* __restrict__ dYt, int ldt) {
  constexpr int BM = 256, BN = 256;
  constexpr int MB = 8, NB = 4;
  __shared__ u32x4 lds[2][2][BM * 8];
  __shared__ float s_part[4][BM];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int G_in = d_in / G;
  const int tiles_n = (d_in + BN - 1) / BN;
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int tm = bid / tiles_n, tn = bid % tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;

  const bool stageA = tid < 256;
  const int sidx = tid & 255;
  const int a = sidx & 7, c = sidx >> 3;
  const int nk = (T + BK - 1) / BK;

  const uint16_t* src = stageA ? dY : X;
  const int ld = stageA ? d_out : d_in;
  const int col0 = (stageA ? m0 : n0) + 8 * c;
  const bool colok = col0 < ld;
  const bool write_t = stageA && dYt != nullptr && tn == 0 && colok;

  f32x4 acc[MB][NB];
  zero_acc(acc);
  u32x4 v[8], tr[8];

  auto gload = [&](int k0) {
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int t = k0 + 8 * a + r;
      v[r] = (colok && t < T) ? ld16(src + int64_t(t) * ld + col0) : zero16();
    }
  };
  auto sstore = [&](int buf, int k0) {
    store_transposed(lds[buf][stageA ? 0 : 1], c, a, v, tr);
    if (write_t && k0 + 8 * a < ldt) {
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) st16(dYt + int64_t(col0 + cc) * ldt + k0 + 8 * a, tr[cc]);
    }
  };

  gload(0);
  sstore(0, 0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) gload((kt + 1) * BK);
    mma_stage<MB, NB>(lds[kt & 1][0], lds[kt & 1][1], wm * 128, wn * 64, lane, acc);
    if (kt + 1 < nk) sstore((kt + 1) & 1, (kt + 1) * BK);
    __syncthreads();
  }

  // Epilogue: multiply by W and reduce each row over this wave's 64 columns
  // (in registers over the 4 column blocks, then across the 16 lanes).
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = wm * 128 + mb * 16 + 4 * (lane >> 4) + j;
      const int o = m0 + r;
      float s = 0.0f;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int i = n0 + wn * 64 + nb * 16 + (lane & 15);
        const float w = (o < d_out && i < d_in) ? bf16_to_f32(W[int64_t(o) * d_in + i]) : 0.0f;
        s += acc[mb][nb][j] * w;
      }
      s += __shfl_xor(s, 1);
      s += __shfl_xor(s, 2);
      s += __shfl_xor(s, 4);
      s += __shfl_xor(s, 8);
      if ((lane & 15) == 0) s_part[wn][r] = s;
    }
  __syncthreads();
  // Combine the four 64-column partials of each row in a fixed order.
  if (tid < BM) {
    const int o = m0 + tid;
    if (o < d_out) {
      float* drow = dgate + int64_t(o) * G_in;
      if constexpr (G == 512) {
        const float h = s_part[0][tid] + s_part[1][tid] + s_part[2][tid] + s_part[3][tid];
        atomicAdd(drow + n0 / 512, h);
      } else if constexpr (G == 256) {
        drow[n0 / 256] = s_part[0][tid] + s_part[1][tid] + s_part[2][tid] + s_part[3][tid];
      } else if constexpr (G == 128) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int gv = n0 / 128 + q;
          if (gv < G_in) drow[gv] = s_part[2 * q][tid] + s_part[2 * q + 1][tid];
        }
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int gv = n0 / 64 + q;
          if (gv < G_in) drow[gv] = s_part[q][tid];
        }
      }
    }
  }
}

// Fill n floats with zero (used before an order-independent accumulation).
__global__ __launch_bounds__(256) void zero_f32_kernel(float* __restrict__ p, int64_t n) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0.0f;
}

// ============================================================================ dX

// Tile: 256 tokens x BN columns of one group column v (BN = min(g, 256));
// K = the kept rows of column v.  Waves (8 / (BN/64)) x (BN/64), wave tile
// (256 / waves_m) x 64.
template <int BN>
__global__ __launch_bounds__(512) void dx_kernel(const uint16_t* __restrict__ dYt, int ldt,
                                                 const uint16_t* __restrict__ W, const int* __restrict__ colcount,
                                                 const int* __restrict__ rows, const float* __restrict__ scales,
                                                 int T, int d_in, int d_out, int g, uint16_t* __restrict__ dX) {
  constexpr int BM = 256;
  constexpr int WAVES_N = BN / 64;
  constexpr int WAVES_M = 8 / WAVES_N;
  constexpr int WTM = BM / WAVES_M;
  constexpr int MB = WTM / 16, NB = 4;
  __shared__ u32x4 As[2][BM * 8];
  __shared__ u32x4 Bs[2][BN * 8];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  const int tiles_n = d_in / BN;
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int tm = bid / tiles_n, tn = bid % tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;
  const int v = n0 / g;
  const int kv = colcount[v];
  const int* __restrict__ rl = rows + int64_t(v) * d_out;
  const float* __restrict__ sl = scales + int64_t(v) * d_out;

  const bool stageA = tid < 256;
  const int sidx = stageA ? tid : tid - 256;
  const int a = sidx & 7, c = sidx >> 3;
  const bool active = stageA || sidx < BN;  // B needs BN staging threads
  const int col0 = stageA ? m0 + 8 * c : n0 + 8 * c;
  const bool colok = stageA ? col0 < T : true;

  f32x4 acc[MB][NB];
  zero_acc(acc);
  u32x4 v8[8], tr[8];
  const int nk = (kv + BK - 1) / BK;

  auto gload = [&](int k0) {
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int kidx = k0 + 8 * a + r;
      v8[r] = zero16();
      if (active && colok && kidx < kv) {
        const int o = rl[kidx];
        if (stageA) {
          v8[r] = ld16(dYt + int64_t(o) * ldt + col0);
        } else {
          const float s = sl[kidx];
          u32x4 w = ld16(W + int64_t(o) * d_in + col0);
          v8[r] = s == 1.0f ? w : scale_bf16x8(w, s);
        }
      }
    }
  };
  auto sstore = [&](int buf) {
    if (active) store_transposed(stageA ? As[buf] : Bs[buf], c, a, v8, tr);
  };

  if (nk > 0) {
    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      if (kt + 1 < nk) gload((kt + 1) * BK);
      mma_stage<MB, NB>(As[kt & 1], Bs[kt & 1], wm * WTM, wn * 64, lane, acc);
      if (kt + 1 < nk) sstore((kt + 1) & 1);
      __syncthreads();
    }
  }
  store_bf16_tile<MB, NB>(acc, dX, d_in, m0 + wm * WTM, n0 + wn * 64, T, d_in, lane);
}

// ============================================================================ fwd

// Tile: 256 tokens x 256 output rows; K walks the group columns that at least
// one row of the tile keeps, G/64 stages per column.  Waves 2 (t) x 4 (o),
// wave tile 128 x 64.  Operands are K-contiguous in HBM, staged directly.
template <int G>
__global__ __launch_bounds__(512) void fwd_kernel(const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
                                                  const float* __restrict__ mask, int T, int d_in, int d_out,
                                                  uint16_t* __restrict__ Y) {
  constexpr int BM = 256, BN = 256, MB = 8, NB = 4;
  constexpr int SUB = G / BK;  // stages per group column
  constexpr int MAXG = 512;    // G_in limit (checked by the host)
  __shared__ u32x4 As[2][BM * 8];
  __shared__ u32x4 Bs[2][BN * 8];
  __shared__ int s_flag[MAXG];
  __shared__ int s_cols[MAXG];
  __shared__ int s_ncols;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int G_in = d_in / G;
  const int tiles_n = (d_out + BN - 1) / BN;
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int tm = bid / tiles_n, tn = bid % tiles_n;
  const int m0 = tm * BM, n0 = tn * BN;

  // Group columns kept by at least one row of this tile, in increasing order.
  for (int q = tid; q < G_in; q += 512) s_flag[q] = 0;
  __syncthreads();
  const int nrows = min(BN, d_out - n0);
  for (int idx = tid; idx < nrows * G_in; idx += 512)
    if (mask[int64_t(n0) * G_in + idx] != 0.0f) s_flag[idx % G_in] = 1;
  __syncthreads();
  if (wave == 0) {
    int cnt = 0;
    for (int vb = 0; vb < G_in; vb += 64) {
      const bool f = vb + lane < G_in && s_flag[vb + lane];
      const uint64_t bal = __ballot(f);
      if (f) s_cols[cnt + __popcll(bal & ((uint64_t(1) << lane) - 1))] = vb + lane;
      cnt += __popcll(bal);
    }
    if (lane == 0) s_ncols = cnt;
  }
  __syncthreads();
  const int nst = s_ncols * SUB;

  f32x4 acc[MB][NB];
  zero_acc(acc);
  u32x4 xa[4], wb[4];

  // Staging: each thread moves four 16-byte chunks of each operand per stage.
  auto gload = [&](int st) {
    const int v = s_cols[st / SUB];
    const int k0 = v * G + (st % SUB) * BK;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = tid + 512 * q;
      const int row = idx >> 3, kc = idx & 7;
      const int t = m0 + row;
      xa[q] = t < T ? ld16(X + int64_t(t) * d_in + k0 + 8 * kc) : zero16();
      const int o = n0 + row;
      const float m = o < d_out ? mask[int64_t(o) * G_in + v] : 0.0f;
      wb[q] = zero16();
      if (m != 0.0f) {
        const u32x4 w = ld16(W + int64_t(o) * d_in + k0 + 8 * kc);
        wb[q] = m == 1.0f ? w : scale_bf16x8(w, m);
      }
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = tid + 512 * q;
      const int row = idx >> 3, kc = idx & 7;
      As[buf][swz64(row, kc)] = xa[q];
      Bs[buf][swz64(row, kc)] = wb[q];
    }
  };

  if (nst > 0) {
    gload(0);
    sstore(0);
    __syncthreads();
    for (int st = 0; st < nst; ++st) {
      if (st + 1 < nst) gload(st + 1);
      mma_stage<MB, NB>(As[st & 1], Bs[st & 1], wm * 128, wn * 64, lane, acc);
      if (st + 1 < nst) sstore((st + 1) & 1);
      __syncthreads();
    }
  }
  store_bf16_tile<MB, NB>(acc, Y, d_out, m0 + wm * 128, n0 + wn * 64, T, d_out, lane);
}

// ============================================================================ dY^T

// Standalone transpose dY [T, d_out] -> dYt [d_out, ldt] for a backward that
// computes dX without dgate.  One 8 x 8 block per thread; t in [T, ldt) is zero.
__global__ __launch_bounds__(256) void transpose_kernel(const uint16_t* __restrict__ dY, int T, int d_out,
                                                        uint16_t* __restrict__ dYt, int ldt) {
  const int tchunks = ldt / 8;
  const int64_t blk = int64_t(blockIdx.x) * 256 + threadIdx.x;
  const int64_t nblk = int64_t(tchunks) * (d_out / 8);
  if (blk >= nblk) return;
  const int a = int(blk % tchunks);  // token chunk
  const int c = int(blk / tchunks);  // output-row chunk
  u32x4 v[8], tr[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int t = 8 * a + r;
    v[r] = t < T ? ld16(dY + int64_t(t) * d_out + 8 * c) : zero16();
  }
  transpose8x8_b16(v, tr);
#pragma unroll
  for (int cc = 0; cc < 8; ++cc) st16(dYt + int64_t(8 * c + cc) * ldt + 8 * a, tr[cc]);
}

// ============================================================================ launchers

hipError_t launch_dgate(const uint16_t* dY, const uint16_t* X, const uint16_t* W, int T, int d_in, int d_out, int g,
                        float* dgate, uint16_t* dYt, int ldt, hipStream_t s) {
  const int tiles = ((d_out + 255) / 256) * ((d_in + 255) / 256);
  if (g == 512) {
    const int64_t n = int64_t(d_out) * (d_in / g);
    hipLaunchKernelGGL(zero_f32_kernel, dim3(unsigned(n / 256 + 1 < 4096 ? n / 256 + 1 : 4096)), dim3(256), 0, s,
                       dgate, n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  switch (g) {
    case 64: hipLaunchKernelGGL(dgate_kernel<64>, dim3(tiles), dim3(512), 0, s, dY, X, W, T, d_in, d_out, dgate, dYt, ldt); break;
    case 128: hipLaunchKernelGGL(dgate_kernel<128>, dim3(tiles), dim3(512), 0, s, dY, X, W, T, d_in, d_out, dgate, dYt, ldt); break;
    case 256: hipLaunchKernelGGL(dgate_kernel<256>, dim3(tiles), dim3(512), 0, s, dY, X, W, T, d_in, d_out, dgate, dYt, ldt); break;
    case 512: hipLaunchKernelGGL(dgate_kernel<512>, dim3(tiles), dim3(512), 0, s, dY, X, W, T, d_in, d_out, dgate, dYt, ldt); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_transpose(const uint16_t* dY, int T, int d_out, uint16_t* dYt, int ldt, hipStream_t s) {
  const int64_t nblk = int64_t(ldt / 8) * (d_out / 8);
  hipLaunchKernelGGL(transpose_kernel, dim3(unsigned((nblk + 255) / 256)), dim3(256), 0, s, dY, T, d_out, dYt, ldt);
  return hipGetLastError();
}

hipError_t launch_dx(const uint16_t* dYt, int ldt, const uint16_t* W, const int* colcount, const int* rows,
                     const float* scales, int T, int d_in, int d_out, int g, uint16_t* dX, hipStream_t s) {
  const int bn = g < 256 ? g : 256;
  const int tiles = ((T + 255) / 256) * (d_in / bn);
  switch (bn) {
    case 64: hipLaunchKernelGGL(dx_kernel<64>, dim3(tiles), dim3(512), 0, s, dYt, ldt, W, colcount, rows, scales, T, d_in, d_out, g, dX); break;
    case 128: hipLaunchKernelGGL(dx_kernel<128>, dim3(tiles), dim3(512), 0, s, dYt, ldt, W, colcount, rows, scales, T, d_in, d_out, g, dX); break;
    case 256: hipLaunchKernelGGL(dx_kernel<256>, dim3(tiles), dim3(512), 0, s, dYt, ldt, W, colcount, rows, scales, T, d_in, d_out, g, dX); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_fwd(const uint16_t* X, const uint16_t* W, const float* mask, int T, int d_in, int d_out, int g,
                      uint16_t* Y, hipStream_t s) {
  const int tiles = ((T + 255) / 256) * ((d_out + 255) / 256);
  switch (g) {
    case 64: hipLaunchKernelGGL(fwd_kernel<64>, dim3(tiles), dim3(512), 0, s, X, W, mask, T, d_in, d_out, Y); break;
    case 128: hipLaunchKernelGGL(fwd_kernel<128>, dim3(tiles), dim3(512), 0, s, X, W, mask, T, d_in, d_out, Y); break;
    case 256: hipLaunchKernelGGL(fwd_kernel<256>, dim3(tiles), dim3(512), 0, s, X, W, mask, T, d_in, d_out, Y); break;
    case 512: hipLaunchKernelGGL(fwd_kernel<512>, dim3(tiles), dim3(512), 0, s, X, W, mask, T, d_in, d_out, Y); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace gm
