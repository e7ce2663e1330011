// Hypernetwork of the mask learner (Sec. 2.2, Eq. 3) and its AdamW step (Table 5).
//
//   o_l      = [GRU_fwd(z_1..z_l); GRU_bwd(z_L..z_l)]        (bidirectional GRU, H units per direction)
//   logit[e] = A[e] . o_{l(e)} + c[e]                       (layer-specific affine heads, rows of one
//                                                            [sum G, 2H] matrix in flat selector order)
//
// The GRU is tiny and sequential over the L layers; the heads hold one row of
// 2H weights per selector (25.3 M rows for LLaMA-2-7B) and are the HBM-bound
// part: the forward reads A once, and the backward reads A with its two AdamW
// moments and writes all three back in one pass, which also accumulates
// do_l = A^T dlogit (with the weights before the update) for the GRU backward.
//
// Work split:
//   gru_input_kernel   W_ih z_l + b_ih for every layer and direction (parallel)
//   gru_fwd_kernel<H>  one block per direction, the recurrence; caches the gates
//   chunk_table_kernel cuts every layer's rows into chunks of kHeadRows, so that a
//                      head block never straddles two layers
//   head_fwd_kernel    logits, one wave row group per selector row
//   head_bwd_kernel    AdamW on A and c, chunk partials of do
//   head_do_kernel     do_l = sum of its chunks' partials, in chunk order
//   gru_bwd_kernel<H>  one block per direction, backpropagation through time
//   gru_wgrad_kernel   weight and bias gradients from the per-step gate gradients
//   adamw_kernel       AdamW over a flat parameter vector (the GRU's)
// Every reduction runs in a fixed order, so results are deterministic.
#include "gm_device.h"
#include "gm_launch.h"

#include <math.h>

namespace gm {

constexpr int kHeadRows = 2048;  // selector rows per head block

__device__ __forceinline__ float sigmoidf(float x) { return 1.0f / (1.0f + expf(-x)); }

// ---------------------------------------------------------------- GRU forward

// gi[dir][l][i] = b_ih[i] + W_ih[i, :] . z[l]
__global__ __launch_bounds__(256) void gru_input_kernel(const float* __restrict__ z, const float* __restrict__ gru,
                                                       int L, int D, int H, float* __restrict__ gi) {
  const int G3 = 3 * H;
  const int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (e >= int64_t(2) * L * G3) return;
  const int i = int(e % G3);
  const int l = int((e / G3) % L);
  const int dir = int(e / (int64_t(L) * G3));
  const float* p = gru + int64_t(dir) * G3 * (D + H + 2);
  const float* w = p + int64_t(i) * D;
  float a = p[int64_t(G3) * (D + H) + i];
  for (int j = 0; j < D; ++j) a += w[j] * z[int64_t(l) * D + j];
  gi[e] = a;
}

// One block per direction; thread i < 3H owns gate row i of W_hh (in
// registers).  cache[dir][l] = (h_prev, r, u, n, W_hn h_prev + b_hn), each H.
// The hidden state is double-buffered in LDS (two barriers per step), and the
// input part of the next step's gates is loaded while this step runs.
template <int H>
__global__ __launch_bounds__(3 * H) void gru_fwd_kernel(const float* __restrict__ gi, const float* __restrict__ gru,
                                                        int L, int D, float* __restrict__ o,
                                                        float* __restrict__ cache) {
  constexpr int G3 = 3 * H;
  __shared__ float s_h[2][H], s_gh[G3];
  const int dir = blockIdx.x, i = threadIdx.x;
  const float* p = gru + int64_t(dir) * G3 * (D + H + 2);
  const float* Whh = p + int64_t(G3) * D;
  const float bh = p[int64_t(G3) * (D + H) + G3 + i];
  float w[H];
#pragma unroll
  for (int k = 0; k < H; ++k) w[k] = Whh[i * H + k];
  auto gates_in = [&](int s, float (&x)[3]) {  // input part of step s's gates for unit i < H
    const int l = dir == 0 ? s : L - 1 - s;
    const float* g = gi + (int64_t(dir) * L + l) * G3;
    x[0] = g[i];
    x[1] = g[H + i];
    x[2] = g[2 * H + i];
  };
  float xg[3] = {0.0f, 0.0f, 0.0f};
  if (i < H) {
    s_h[0][i] = 0.0f;
    gates_in(0, xg);
  }
  __syncthreads();
  for (int s = 0; s < L; ++s) {
    const int l = dir == 0 ? s : L - 1 - s;
    const float* hcur = s_h[s & 1];
    float a = bh;
#pragma unroll
    for (int k = 0; k < H; ++k) a += w[k] * hcur[k];
    s_gh[i] = a;
    __syncthreads();
    if (i < H) {
      float xn[3] = {0.0f, 0.0f, 0.0f};
      if (s + 1 < L) gates_in(s + 1, xn);
      const float r = sigmoidf(xg[0] + s_gh[i]);
      const float u = sigmoidf(xg[1] + s_gh[H + i]);
      const float ghn = s_gh[2 * H + i];
      const float n = tanhf(xg[2] + r * ghn);
      const float hp = hcur[i];
      const float hn = (1.0f - u) * n + u * hp;
      float* c = cache + (int64_t(dir) * L + l) * 5 * H;
      c[i] = hp;
      c[H + i] = r;
      c[2 * H + i] = u;
      c[3 * H + i] = n;
      c[4 * H + i] = ghn;
      o[int64_t(l) * 2 * H + dir * H + i] = hn;
      s_h[(s + 1) & 1][i] = hn;  // the other buffer: this step's readers are past the barrier above
      xg[0] = xn[0];
      xg[1] = xn[1];
      xg[2] = xn[2];
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------- heads

// Chunk c covers rows [start, end) of layer lay; layers are cut at multiples
// of kHeadRows from their first row.  count[0] = number of chunks, first[l] =
// first chunk of layer l (first[L] = count).
__global__ __launch_bounds__(256) void chunk_table_kernel(const int64_t* __restrict__ offsets, int L,
                                                         int* __restrict__ lay, int64_t* __restrict__ start,
                                                         int64_t* __restrict__ end, int* __restrict__ first,
                                                         int* __restrict__ count) {
  __shared__ int s_n[256];
  const int tid = threadIdx.x;
  // per-thread totals over a contiguous run of layers, then a block scan
  const int per = (L + 255) / 256;
  const int l0 = min(tid * per, L), l1 = min(l0 + per, L);
  int n = 0;
  for (int l = l0; l < l1; ++l) n += int((offsets[l + 1] - offsets[l] + kHeadRows - 1) / kHeadRows);
  s_n[tid] = n;
  __syncthreads();
  for (int d = 1; d < 256; d <<= 1) {
    const int add = tid >= d ? s_n[tid - d] : 0;
    __syncthreads();
    s_n[tid] += add;
    __syncthreads();
  }
  int c = s_n[tid] - n;
  for (int l = l0; l < l1; ++l) {
    first[l] = c;
    for (int64_t r = offsets[l]; r < offsets[l + 1]; r += kHeadRows, ++c) {
      lay[c] = l;
      start[c] = r;
      end[c] = min(r + int64_t(kHeadRows), offsets[l + 1]);
    }
  }
  if (tid == 255) {
    first[L] = s_n[255];
    count[0] = s_n[255];
  }
}

// LPR = 2H / 4 lanes per row (four weights per lane), RPW = 64 / LPR rows per wave step.
template <int H>
__global__ __launch_bounds__(256) void head_fwd_kernel(const float* __restrict__ A, const float* __restrict__ cb,
                                                       const float* __restrict__ o, const int* __restrict__ lay,
                                                       const int64_t* __restrict__ start,
                                                       const int64_t* __restrict__ end,
                                                       const int* __restrict__ count, float* __restrict__ logits) {
  constexpr int LPR = 2 * H / 4, RPW = 64 / LPR;
  if (int(blockIdx.x) >= count[0]) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l = lay[blockIdx.x];
  const int64_t r0 = start[blockIdx.x], r1 = end[blockIdx.x];
  const int col = (lane % LPR) * 4;
  const f32x4 ov = *reinterpret_cast<const f32x4*>(o + int64_t(l) * 2 * H + col);
  for (int64_t r = r0 + wave * RPW + lane / LPR; r - (lane / LPR) < r1; r += 4 * RPW) {
    float a = 0.0f;
    if (r < r1) {
      const f32x4 w = *reinterpret_cast<const f32x4*>(A + r * 2 * H + col);
      a = w[0] * ov[0] + w[1] * ov[1] + w[2] * ov[2] + w[3] * ov[3];
    }
#pragma unroll
    for (int x = 1; x < LPR; x <<= 1) a += __shfl_xor(a, x);
    if (r < r1 && lane % LPR == 0) logits[r] = a + cb[r];
  }
}

// One AdamW step on a float4 of parameters (decoupled decay, bias-corrected moments).
// The coefficients are formed in fp64 on the host and rounded once (1 - beta
// directly, not from a rounded beta).
struct AdamW {
  float lr, b1, omb1, b2, omb2, eps, decay, bc1, bc2;  // decay = 1 - lr weight_decay; bc = 1 / (1 - beta^t)
  __device__ __forceinline__ float step(float p, float g, float& m, float& v) const {
    m = b1 * m + omb1 * g;
    v = b2 * v + omb2 * g * g;
    return p * decay - lr * (m * bc1) / (sqrtf(v * bc2) + eps);
  }
};

template <int H>
__global__ __launch_bounds__(256) void head_bwd_kernel(const float* __restrict__ dl, float* __restrict__ A,
                                                       float* __restrict__ cb, float* __restrict__ mA,
                                                       float* __restrict__ vA, float* __restrict__ mc,
                                                       float* __restrict__ vc, const float* __restrict__ o,
                                                       const int* __restrict__ lay, const int64_t* __restrict__ start,
                                                       const int64_t* __restrict__ end, const int* __restrict__ count,
                                                       AdamW opt, float* __restrict__ part) {
  constexpr int LPR = 2 * H / 4, RPW = 64 / LPR;
  __shared__ f32x4 s_do[4][64];
  if (int(blockIdx.x) >= count[0]) return;  // uniform across the block
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l = lay[blockIdx.x];
  const int64_t r0 = start[blockIdx.x], r1 = end[blockIdx.x];
  const int col = (lane % LPR) * 4;
  const f32x4 ov = *reinterpret_cast<const f32x4*>(o + int64_t(l) * 2 * H + col);
  f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int64_t r = r0 + wave * RPW + lane / LPR; r < r1; r += 4 * RPW) {
    const float g = dl[r];
    const int64_t at = r * 2 * H + col;
    f32x4 w = *reinterpret_cast<const f32x4*>(A + at);
    f32x4 m = *reinterpret_cast<const f32x4*>(mA + at);
    f32x4 v = *reinterpret_cast<const f32x4*>(vA + at);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      acc[k] += w[k] * g;
      float mk = m[k], vk = v[k];
      w[k] = opt.step(w[k], g * ov[k], mk, vk);
      m[k] = mk;
      v[k] = vk;
    }
    *reinterpret_cast<f32x4*>(A + at) = w;
    *reinterpret_cast<f32x4*>(mA + at) = m;
    *reinterpret_cast<f32x4*>(vA + at) = v;
    if (lane % LPR == 0) {
      float cm = mc[r], cv = vc[r];
      cb[r] = opt.step(cb[r], g, cm, cv);
      mc[r] = cm;
      vc[r] = cv;
    }
  }
  // do partial of this chunk: over the RPW row slots of the wave, then the four waves
#pragma unroll
  for (int x = LPR; x < 64; x <<= 1)
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[k] += __shfl_xor(acc[k], x);
  s_do[wave][lane] = acc;
  __syncthreads();
  if (threadIdx.x < LPR) {
    const f32x4 s = s_do[0][threadIdx.x] + s_do[1][threadIdx.x] + s_do[2][threadIdx.x] + s_do[3][threadIdx.x];
    *reinterpret_cast<f32x4*>(part + int64_t(blockIdx.x) * 2 * H + threadIdx.x * 4) = s;
  }
}

// do[l][k] = sum over the chunks of layer l, in chunk order.
__global__ __launch_bounds__(256) void head_do_kernel(const float* __restrict__ part, const int* __restrict__ first,
                                                     int L, int H2, float* __restrict__ dout) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= L * H2) return;
  const int l = e / H2, k = e % H2;
  float s = 0.0f;
  for (int c = first[l]; c < first[l + 1]; ++c) s += part[int64_t(c) * H2 + k];
  dout[e] = s;
}

// ---------------------------------------------------------------- GRU backward

// One block of 4H threads per direction.  Phase A (threads k < H): the gate
// gradients of step l from dh = do + carried gradient; phase B (all
// threads, four per hidden unit k): dh_prev[k] = u dh + sum_i W_hh[i, k] dgh[i]
// over a quarter of the 3H rows each, combined with two shuffles.  The
// carried gradient alternates between two LDS buffers, so a step needs two
// barriers; the cached gates of the next step are loaded during this one.
// dgi, dgh [dir][l][3H] are kept for the weight gradients.
template <int H>
__global__ __launch_bounds__(4 * H) void gru_bwd_kernel(const float* __restrict__ dout,
                                                        const float* __restrict__ gru, const float* __restrict__ cache,
                                                        int L, int D, float* __restrict__ dgi,
                                                        float* __restrict__ dgh) {
  constexpr int G3 = 3 * H, RPT = G3 / 4;
  __shared__ float s_dh[2][H], s_carry[H], s_g[G3];  // s_dh double-buffered by step parity
  const int dir = blockIdx.x, tid = threadIdx.x;
  const float* Whh = gru + int64_t(dir) * G3 * (D + H + 2) + int64_t(G3) * D;
  const int k = tid >> 2, seg = tid & 3;
  float wc[RPT];  // W_hh[seg * RPT + j, k]
#pragma unroll
  for (int j = 0; j < RPT; ++j) wc[j] = Whh[(seg * RPT + j) * H + k];
  // this unit's cached gates and output gradient of step s, loaded one step ahead
  auto fetch = [&](int s, float (&v)[6]) {
    const int l = dir == 0 ? s : L - 1 - s;
    const float* c = cache + (int64_t(dir) * L + l) * 5 * H;
#pragma unroll
    for (int q = 0; q < 5; ++q) v[q] = c[q * H + tid];
    v[5] = dout[int64_t(l) * 2 * H + dir * H + tid];
  };
  float cur[6] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
  if (tid < H) {
    s_dh[(L - 1) & 1][tid] = 0.0f;
    fetch(L - 1, cur);
  }
  __syncthreads();
  for (int s = L - 1; s >= 0; --s) {
    const int l = dir == 0 ? s : L - 1 - s;
    if (tid < H) {
      float nxt[6] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
      if (s > 0) fetch(s - 1, nxt);
      const float hp = cur[0], r = cur[1], u = cur[2], n = cur[3], ghn = cur[4];
      const float dh = s_dh[s & 1][tid] + cur[5];
      const float dan = dh * (1.0f - u) * (1.0f - n * n);
      const float dar = dan * ghn * r * (1.0f - r);
      const float dau = dh * (hp - n) * u * (1.0f - u);
      float* gi = dgi + (int64_t(dir) * L + l) * G3;
      float* gh = dgh + (int64_t(dir) * L + l) * G3;
      gi[tid] = dar;
      gi[H + tid] = dau;
      gi[2 * H + tid] = dan;
      gh[tid] = dar;
      gh[H + tid] = dau;
      gh[2 * H + tid] = dan * r;
      s_g[tid] = dar;
      s_g[H + tid] = dau;
      s_g[2 * H + tid] = dan * r;
      s_carry[tid] = dh * u;
#pragma unroll
      for (int q = 0; q < 6; ++q) cur[q] = nxt[q];
    }
    __syncthreads();
    float a = 0.0f;
#pragma unroll
    for (int j = 0; j < RPT; ++j) a += wc[j] * s_g[seg * RPT + j];
    a += __shfl_xor(a, 1);
    a += __shfl_xor(a, 2);
    if (seg == 0 && s > 0) s_dh[(s - 1) & 1][k] = s_carry[k] + a;  // the buffer phase A did not read
    __syncthreads();
  }
}

// Weight and bias gradients of one direction, one thread per parameter, sums over l in order:
//   dW_ih[i, j] = sum_l dgi[l][i] z[l][j],  dW_hh[i, k] = sum_l dgh[l][i] h_prev[l][k],
//   db_ih[i] = sum_l dgi[l][i],             db_hh[i] = sum_l dgh[l][i].
__global__ __launch_bounds__(256) void gru_wgrad_kernel(const float* __restrict__ z, const float* __restrict__ cache,
                                                       const float* __restrict__ dgi, const float* __restrict__ dgh,
                                                       int L, int D, int H, float* __restrict__ dgru) {
  const int G3 = 3 * H;
  const int64_t P = int64_t(G3) * (D + H + 2);
  const int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (e >= 2 * P) return;
  const int dir = int(e / P);
  const int64_t q = e % P;
  const float* gi = dgi + int64_t(dir) * L * G3;
  const float* gh = dgh + int64_t(dir) * L * G3;
  const float* hc = cache + int64_t(dir) * L * 5 * H;  // h_prev is the first of the five
  float s = 0.0f;
  if (q < int64_t(G3) * D) {
    const int i = int(q / D), j = int(q % D);
    for (int l = 0; l < L; ++l) s += gi[int64_t(l) * G3 + i] * z[int64_t(l) * D + j];
  } else if (q < int64_t(G3) * (D + H)) {
    const int64_t t = q - int64_t(G3) * D;
    const int i = int(t / H), k = int(t % H);
    for (int l = 0; l < L; ++l) s += gh[int64_t(l) * G3 + i] * hc[int64_t(l) * 5 * H + k];
  } else if (q < int64_t(G3) * (D + H + 1)) {
    const int i = int(q - int64_t(G3) * (D + H));
    for (int l = 0; l < L; ++l) s += gi[int64_t(l) * G3 + i];
  } else {
    const int i = int(q - int64_t(G3) * (D + H + 1));
    for (int l = 0; l < L; ++l) s += gh[int64_t(l) * G3 + i];
  }
  dgru[e] = s;
}

__global__ __launch_bounds__(256) void adamw_kernel(float* __restrict__ p, const float* __restrict__ g,
                                                   float* __restrict__ m, float* __restrict__ v, int64_t n,
                                                   AdamW opt) {
  const int64_t stride = int64_t(gridDim.x) * 256;
  for (int64_t e = int64_t(blockIdx.x) * 256 + threadIdx.x; e < n; e += stride) {
    float mm = m[e], vv = v[e];
    p[e] = opt.step(p[e], g[e], mm, vv);
    m[e] = mm;
    v[e] = vv;
  }
}

// ---------------------------------------------------------------- launchers

int hyper_max_chunks(int64_t G_total, int L) { return int((G_total + kHeadRows - 1) / kHeadRows) + L; }

static AdamW make_adamw(double lr, double b1, double b2, double eps, double wd, int step) {
  AdamW o;
  o.lr = float(lr);
  o.b1 = float(b1);
  o.omb1 = float(1.0 - b1);
  o.b2 = float(b2);
  o.omb2 = float(1.0 - b2);
  o.eps = float(eps);
  o.decay = float(1.0 - lr * wd);
  o.bc1 = float(1.0 / (1.0 - pow(b1, double(step))));
  o.bc2 = float(1.0 / (1.0 - pow(b2, double(step))));
  return o;
}

#define GM_HYPER_H(KERNEL, GRID, BLOCK, ...)                                                            \
  switch (H) {                                                                                          \
    case 32: hipLaunchKernelGGL((KERNEL<32>), dim3(GRID), dim3((BLOCK) * 32), 0, s, __VA_ARGS__); break;   \
    case 64: hipLaunchKernelGGL((KERNEL<64>), dim3(GRID), dim3((BLOCK) * 64), 0, s, __VA_ARGS__); break;   \
    case 128: hipLaunchKernelGGL((KERNEL<128>), dim3(GRID), dim3((BLOCK) * 128), 0, s, __VA_ARGS__); break; \
    default: return hipErrorInvalidValue;                                                               \
  }

hipError_t launch_hyper_fwd(const float* z, const float* gru, const float* A, const float* c, const int64_t* offsets,
                            int L, int D, int H, int64_t G_total, float* logits, const HyperWs& w, hipStream_t s) {
  const int64_t n_in = int64_t(2) * L * 3 * H;
  hipLaunchKernelGGL(gru_input_kernel, dim3(unsigned((n_in + 255) / 256)), dim3(256), 0, s, z, gru, L, D, H, w.gi);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  GM_HYPER_H(gru_fwd_kernel, 2, 3, w.gi, gru, L, D, w.o, w.cache)
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(chunk_table_kernel, dim3(1), dim3(256), 0, s, offsets, L, w.lay, w.start, w.end, w.first,
                     w.count);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const unsigned blocks = unsigned(hyper_max_chunks(G_total, L));
  switch (H) {
    case 32: hipLaunchKernelGGL(head_fwd_kernel<32>, dim3(blocks), dim3(256), 0, s, A, c, w.o, w.lay, w.start, w.end, w.count, logits); break;
    case 64: hipLaunchKernelGGL(head_fwd_kernel<64>, dim3(blocks), dim3(256), 0, s, A, c, w.o, w.lay, w.start, w.end, w.count, logits); break;
    case 128: hipLaunchKernelGGL(head_fwd_kernel<128>, dim3(blocks), dim3(256), 0, s, A, c, w.o, w.lay, w.start, w.end, w.count, logits); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_hyper_bwd(const float* dlogits, const float* z, const float* gru, float* A, float* c, float* mA,
                            float* vA, float* mc, float* vc, int L, int D, int H, int64_t G_total, double lr,
                            double beta1, double beta2, double eps, double weight_decay, int step, float* dgru,
                            const HyperWs& w, hipStream_t s) {
  const AdamW opt = make_adamw(lr, beta1, beta2, eps, weight_decay, step);
  const unsigned blocks = unsigned(hyper_max_chunks(G_total, L));
  switch (H) {
    case 32: hipLaunchKernelGGL(head_bwd_kernel<32>, dim3(blocks), dim3(256), 0, s, dlogits, A, c, mA, vA, mc, vc, w.o, w.lay, w.start, w.end, w.count, opt, w.part); break;
    case 64: hipLaunchKernelGGL(head_bwd_kernel<64>, dim3(blocks), dim3(256), 0, s, dlogits, A, c, mA, vA, mc, vc, w.o, w.lay, w.start, w.end, w.count, opt, w.part); break;
    case 128: hipLaunchKernelGGL(head_bwd_kernel<128>, dim3(blocks), dim3(256), 0, s, dlogits, A, c, mA, vA, mc, vc, w.o, w.lay, w.start, w.end, w.count, opt, w.part); break;
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(head_do_kernel, dim3(unsigned((L * 2 * H + 255) / 256)), dim3(256), 0, s, w.part, w.first, L,
                     2 * H, w.dout);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  GM_HYPER_H(gru_bwd_kernel, 2, 4, w.dout, gru, w.cache, L, D, w.dgi, w.dgh)
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int64_t P2 = int64_t(2) * 3 * H * (D + H + 2);
  hipLaunchKernelGGL(gru_wgrad_kernel, dim3(unsigned((P2 + 255) / 256)), dim3(256), 0, s, z, w.cache, w.dgi, w.dgh,
                     L, D, H, dgru);
  return hipGetLastError();
}

hipError_t launch_adamw(float* p, const float* g, float* m, float* v, int64_t n, double lr, double beta1,
                        double beta2, double eps, double weight_decay, int step, hipStream_t s) {
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(adamw_kernel, dim3(unsigned(blocks < 8192 ? blocks : 8192)), dim3(256), 0, s, p, g, m, v, n,
                     make_adamw(lr, beta1, beta2, eps, weight_decay, step));
  return hipGetLastError();
}

}  // namespace gm
