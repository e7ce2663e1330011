// Sparsity-budget regulariser (Sec. 2.3) over the selectors of L layers
// stored back to back in one flat array: layer l owns [offsets[l], offsets[l+1]).
//
//   kept^l = #{ mask != 0 } in layer l                    (integer, exact)
//   s^l    = 1 - kept^l / G^l,  s = sum_l s^l P^l / sum_l P^l   (Eq. 2)
//   global : L = lambda |log(s / s_t)|,            c^l = lambda sgn(log(s/s_t)) / s * (-(P^l / G^l) / sum P)
//   uniform: L = sum_l lambda |log(s^l / s_t)|,    c^l = lambda sgn(log(s^l/s_t)) / s^l * (-1 / G^l)
//
// c^l is the derivative of L with respect to every selector of layer l; the
// STE backward folds it into the logit gradient:
//   dlogit = (dgate + c^l) * y (1 - y) / tau.
//
// Three passes: a segmented count over the flat mask (4 bytes per group, HBM
// bound), a one-block finalize in fp64, and the folded gate backward (12
// bytes per group).  A block owns a contiguous chunk of kChunk groups, so it
// meets at most a few layer boundaries; it counts each layer it touches with
// one block reduction and one 64-bit atomic.
#include "gm_device.h"
#include "gm_launch.h"

namespace gm {

constexpr int kBudgetThreads = 256;
constexpr int kPerThread = 16;                                // groups per thread (four float4)
constexpr int64_t kChunk = int64_t(kBudgetThreads) * kPerThread;  // groups per block

// Layer of group e: the largest l in [lo, hi] with offsets[l] <= e (offsets
// nondecreasing; out-of-order offsets give a wrong layer, never a wrong address).
__device__ __forceinline__ int layer_of(const int64_t* __restrict__ offsets, int lo, int hi, int64_t e) {
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (offsets[mid] <= e) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__global__ __launch_bounds__(256) void fill_u64_kernel(unsigned long long* __restrict__ p, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0ull;
}

__device__ __forceinline__ int block_sum_int(int v, int* s_red) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d);
  const int wave = threadIdx.x >> 6;
  __syncthreads();  // s_red is reused across calls
  if ((threadIdx.x & 63) == 0) s_red[wave] = v;
  __syncthreads();
  return s_red[0] + s_red[1] + s_red[2] + s_red[3];
}

__global__ __launch_bounds__(kBudgetThreads) void count_kept_kernel(const float* __restrict__ mask, int64_t n,
                                                                   const int64_t* __restrict__ offsets, int L,
                                                                   unsigned long long* __restrict__ kept) {
  __shared__ int s_red[4];
  const int64_t start = int64_t(blockIdx.x) * kChunk;
  const int64_t end = min(start + kChunk, n);
  // Groups of this thread: four float4 at start + 4 (t + 256 q), q = 0..3.
  float v[kPerThread];
  int64_t e0[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    e0[q] = start + 4 * (int64_t(threadIdx.x) + kBudgetThreads * q);
    if (e0[q] + 4 <= end) {
      const float4 f = *reinterpret_cast<const float4*>(mask + e0[q]);
      v[4 * q + 0] = f.x; v[4 * q + 1] = f.y; v[4 * q + 2] = f.z; v[4 * q + 3] = f.w;
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) v[4 * q + k] = e0[q] + k < end ? mask[e0[q] + k] : 0.0f;
    }
  }
  const int lo = layer_of(offsets, 0, L - 1, start);
  const int hi = layer_of(offsets, lo, L - 1, end - 1);
  for (int l = lo; l <= hi; ++l) {
    const int64_t a = max(start, offsets[l]);
    const int64_t b = l + 1 < L ? min(end, offsets[l + 1]) : end;
    int c = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int64_t e = e0[q] + k;
        c += (e >= a && e < b && v[4 * q + k] != 0.0f) ? 1 : 0;
      }
    const int total = block_sum_int(c, s_red);
    if (threadIdx.x == 0 && total) atomicAdd(kept + l, (unsigned long long)total);
  }
}

// One block of 256 threads.  Sums run in a fixed tree order, so the result is
// deterministic.
__global__ __launch_bounds__(256) void budget_finalize_kernel(const unsigned long long* __restrict__ kept,
                                                              const int64_t* __restrict__ offsets,
                                                              const int64_t* __restrict__ params, int L,
                                                              double s_t, double lam, int uniform,
                                                              double* __restrict__ loss, float* __restrict__ coeff) {
  __shared__ double s_a[256], s_b[256];
  const int tid = threadIdx.x;
  // global: a = sum_l s^l P^l written as the pruned weight count (G^l - kept^l) P^l / G^l,
  // exact in fp64 when G^l divides P^l (whole groups), b = sum_l P^l, s = a / b rounded once;
  // uniform: a = sum_l lambda |log(s^l / s_t)| with s^l = (G^l - kept^l) / G^l rounded once.
  double a = 0.0, b = 0.0;
  for (int l = tid; l < L; l += 256) {
    const int64_t Gl = offsets[l + 1] - offsets[l];
    const double G = double(Gl);
    const double pruned = double(Gl - int64_t(kept[l]));
    if (uniform) {
      a += lam * fabs(log((pruned / G) / s_t));
    } else {
      a += pruned * double(params[l]) / G;
      b += double(params[l]);
    }
  }
  s_a[tid] = a;
  s_b[tid] = b;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if (tid < w) {
      s_a[tid] += s_a[tid + w];
      s_b[tid] += s_b[tid + w];
    }
    __syncthreads();
  }
  const double A = s_a[0], B = s_b[0];
  const double s = uniform ? 0.0 : A / B;
  for (int l = tid; l < L; l += 256) {
    const double G = double(offsets[l + 1] - offsets[l]);
    double c;
    if (uniform) {
      const double sl = double(offsets[l + 1] - offsets[l] - int64_t(kept[l])) / G;
      const double r = log(sl / s_t);
      const double sg = r > 0.0 ? 1.0 : (r < 0.0 ? -1.0 : 0.0);
      c = lam * sg / sl * (-1.0 / G);
    } else {
      const double r = log(s / s_t);
      const double sg = r > 0.0 ? 1.0 : (r < 0.0 ? -1.0 : 0.0);
      c = lam * sg / s * (-(double(params[l]) / G) / B);
    }
    coeff[l] = float(c);
  }
  if (tid == 0) *loss = uniform ? A : lam * fabs(log(s / s_t));
}

// dlogits may alias dgate: every element is read before the same thread writes it.
__global__ __launch_bounds__(kBudgetThreads) void gate_bwd_budget_kernel(const float* dgate,
                                                                        const float* __restrict__ soft, int64_t n,
                                                                        float tau,
                                                                        const int64_t* __restrict__ offsets, int L,
                                                                        const float* __restrict__ coeff,
                                                                        float* dlogits) {
  const int64_t start = int64_t(blockIdx.x) * kChunk;
  const int64_t end = min(start + kChunk, n);
  const int lo = layer_of(offsets, 0, L - 1, start);
  const int hi = layer_of(offsets, lo, L - 1, end - 1);
  const float c_lo = coeff[lo];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t e0 = start + 4 * (int64_t(threadIdx.x) + kBudgetThreads * q);
    if (e0 >= end) continue;
    float d[4], y[4], c[4];
    const bool full = e0 + 4 <= end;
    if (full) {
      const float4 df = *reinterpret_cast<const float4*>(dgate + e0);
      const float4 yf = *reinterpret_cast<const float4*>(soft + e0);
      d[0] = df.x; d[1] = df.y; d[2] = df.z; d[3] = df.w;
      y[0] = yf.x; y[1] = yf.y; y[2] = yf.z; y[3] = yf.w;
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        d[k] = e0 + k < end ? dgate[e0 + k] : 0.0f;
        y[k] = e0 + k < end ? soft[e0 + k] : 0.0f;
      }
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) c[k] = lo == hi ? c_lo : coeff[layer_of(offsets, lo, hi, e0 + k)];
    float r[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) r[k] = (d[k] + c[k]) * y[k] * (1.0f - y[k]) / tau;
    if (full) {
      __builtin_nontemporal_store(f32x4{r[0], r[1], r[2], r[3]}, reinterpret_cast<f32x4*>(dlogits + e0));  // streamed
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k)
        if (e0 + k < end) dlogits[e0 + k] = r[k];
    }
  }
}

static unsigned chunk_grid(int64_t n) { return unsigned((n + kChunk - 1) / kChunk); }

hipError_t launch_budget_loss(const float* mask, int64_t n, const int64_t* offsets, const int64_t* params, int L,
                              float s_target, float lambda, int uniform, unsigned long long* kept, double* loss,
                              float* coeff, hipStream_t s) {
  hipLaunchKernelGGL(fill_u64_kernel, dim3(unsigned((L + 255) / 256 < 64 ? (L + 255) / 256 : 64)), dim3(256), 0, s,
                     kept, L);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(count_kept_kernel, dim3(chunk_grid(n)), dim3(kBudgetThreads), 0, s, mask, n, offsets, L, kept);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(budget_finalize_kernel, dim3(1), dim3(256), 0, s, kept, offsets, params, L, double(s_target),
                     double(lambda), uniform, loss, coeff);
  return hipGetLastError();
}

hipError_t launch_gate_bwd_budget(const float* dgate, const float* soft, int64_t n, float tau,
                                  const int64_t* offsets, int L, const float* coeff, float* dlogits, hipStream_t s) {
  hipLaunchKernelGGL(gate_bwd_budget_kernel, dim3(chunk_grid(n)), dim3(kBudgetThreads), 0, s, dgate, soft, n, tau,
                     offsets, L, coeff, dlogits);
  return hipGetLastError();
}

}  // namespace gm
