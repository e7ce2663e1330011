// Group index structures built from a selector matrix mask [d_out / g_out, G_in]
// (g_out x g groups; output row o belongs to mask row o / g_out).
//
// Column lists (consumed by the dX GEMM): list column c covers nsub
// consecutive group columns (nsub = 1 unless groups are narrower than 64
// columns).  For every c: the output rows that keep one of its groups, in
// increasing order, rows[c * d_out + j], with their mask values
// scales[(c * d_out + j) * nsub + s] for group column c * nsub + s, their kept
// bits subbits[c * d_out + j] (bit s; written only when nsub > 1), the count
// colcount[c] and colsoft[c] = 1 when some kept value differs from 1.  This
// is the group-compacted view of W that lets the dX K-loop visit only kept
// groups.
//
// Row-packed export (Appendix F): rowptr / packed values / group column ids,
// written by three passes (count per row, scan, copy).
#include "gm_device.h"
#include "gm_launch.h"

namespace gm {

// One 1024-thread block per list column c.  The rows go in chunks of 4096:
// thread t owns rows 4t .. 4t + 3 of the chunk and loads all of their
// selectors before any of them is used (one memory round trip per chunk, not
// one per 1024 rows), counts its kept rows, and finds where they go with a
// block-wide exclusive scan of the counts (a shuffle scan inside each wave,
// then the 16 wave totals in LDS).  Rows stay in increasing order.
constexpr int kListRowsPerThread = 4;

__global__ __launch_bounds__(1024) void col_lists_kernel(const float* __restrict__ mask, int d_out, int G_in,
                                                        int go, int nsub, int* __restrict__ colcount,
                                                        int* __restrict__ colsoft, int* __restrict__ rows,
                                                        float* __restrict__ scales, int* __restrict__ subbits) {
  constexpr int R = kListRowsPerThread;
  const int c = blockIdx.x;
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  __shared__ int wave_tot[16];
  __shared__ int s_soft;
  if (threadIdx.x == 0) s_soft = 0;
  bool soft = false;
  int base = 0;
  for (int o0 = 0; o0 < d_out; o0 += 1024 * R) {
    const int ob = o0 + int(threadIdx.x) * R;
    float m[R][4];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        m[r][q] = (q < nsub && ob + r < d_out) ? mask[int64_t((ob + r) / go) * G_in + c * nsub + q] : 0.0f;
    int bits[R];
    int cnt = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
      bits[r] = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        bits[r] |= int(m[r][q] != 0.0f) << q;
        soft |= m[r][q] != 0.0f && m[r][q] != 1.0f;
      }
      cnt += bits[r] != 0;
    }
    // inclusive scan of the counts within the wave
    int inc = cnt;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int up = __shfl_up(inc, d);
      if (lane >= d) inc += up;
    }
    if (lane == 63) wave_tot[w] = inc;
    __syncthreads();
    int off = base + inc - cnt;
    int chunk_total = 0;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int t = wave_tot[q];
      if (q < w) off += t;
      chunk_total += t;
    }
#pragma unroll
    for (int r = 0; r < R; ++r)
      if (bits[r]) {
        const int64_t e = int64_t(c) * d_out + off;
        rows[e] = ob + r;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (q < nsub) scales[e * nsub + q] = m[r][q];
        if (nsub > 1) subbits[e] = bits[r];
        ++off;
      }
    base += chunk_total;
    __syncthreads();  // wave_tot is rewritten by the next chunk
  }
  if (soft) s_soft = 1;
  __syncthreads();
  if (threadIdx.x == 0) {
    colcount[c] = base;
    colsoft[c] = s_soft;
  }
}

hipError_t launch_col_lists(const float* mask, int d_out, int G_in, int go, int nsub, int* colcount, int* colsoft,
                            int* rows, float* scales, int* subbits, hipStream_t s) {
  hipLaunchKernelGGL(col_lists_kernel, dim3(G_in / nsub), dim3(1024), 0, s, mask, d_out, G_in, go, nsub, colcount,
                     colsoft, rows, scales, subbits);
  return hipGetLastError();
}

// ------------------------------------------------------------------ row packing

// rowptr[o + 1] = number of kept groups of row o; rowptr[0] = 0.
__global__ __launch_bounds__(256) void row_counts_kernel(const float* __restrict__ mask, int d_out, int G_in,
                                                         int go, int* __restrict__ rowptr) {
  const int o = blockIdx.x * blockDim.x + threadIdx.x;
  if (o == 0) rowptr[0] = 0;
  if (o >= d_out) return;
  int c = 0;
  for (int v = 0; v < G_in; ++v) c += mask[int64_t(o / go) * G_in + v] != 0.0f;
  rowptr[o + 1] = c;
}

// In-place inclusive scan of rowptr[1 .. d_out] by one 1024-thread block: each
// thread scans a contiguous run serially, the run totals are scanned in LDS.
__global__ __launch_bounds__(1024) void scan_rowptr_kernel(int* __restrict__ rowptr, int d_out) {
  __shared__ int tot[1024];
  const int per = (d_out + 1023) / 1024;
  const int beg = 1 + threadIdx.x * per;
  const int end = min(beg + per, d_out + 1);
  int s = 0;
  for (int i = beg; i < end; ++i) s += rowptr[i];
  tot[threadIdx.x] = s;
  __syncthreads();
  for (int d = 1; d < 1024; d <<= 1) {
    const int add = threadIdx.x >= d ? tot[threadIdx.x - d] : 0;
    __syncthreads();
    tot[threadIdx.x] += add;
    __syncthreads();
  }
  int run = threadIdx.x ? tot[threadIdx.x - 1] : 0;
  for (int i = beg; i < end; ++i) {
    run += rowptr[i];
    rowptr[i] = run;
  }
}

// One wave per row: copies each kept group (g bf16 values of the row) to its
// packed slot; a g_out x g group becomes g_out row pieces.
__global__ __launch_bounds__(256) void pack_copy_kernel(const uint16_t* __restrict__ W,
                                                        const float* __restrict__ mask, int d_in, int d_out,
                                                        int g, int go, int64_t capacity, const int* __restrict__ rowptr,
                                                        uint16_t* __restrict__ Wp, int* __restrict__ chunk,
                                                        float* __restrict__ scale) {
  const int lane = threadIdx.x & 63;
  const int o = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (o >= d_out) return;
  const int G_in = d_in / g;
  int64_t j = rowptr[o];
  const int vec_per_group = g / 8;  // 16-byte vectors per group
  for (int v = 0; v < G_in; ++v) {
    const float m = mask[int64_t(o / go) * G_in + v];
    if (m == 0.0f) continue;  // uniform across the wave
    if (j < capacity) {
      const uint16_t* src = W + int64_t(o) * d_in + int64_t(v) * g;
      uint16_t* dst = Wp + j * g;
      for (int q = lane; q < vec_per_group; q += 64) st16(dst + q * 8, ld16(src + q * 8));
      if (lane == 0) {
        chunk[j] = v;
        scale[j] = m;
      }
    }
    ++j;
  }
}

hipError_t launch_pack_rows(const uint16_t* W, const float* mask, int d_in, int d_out, int g, int go,
                            int64_t capacity, uint16_t* Wp, int* chunk, float* scale, int* rowptr, hipStream_t s) {
  const int G_in = d_in / g;
  hipLaunchKernelGGL(row_counts_kernel, dim3((d_out + 255) / 256), dim3(256), 0, s, mask, d_out, G_in, go, rowptr);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(scan_rowptr_kernel, dim3(1), dim3(1024), 0, s, rowptr, d_out);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(pack_copy_kernel, dim3((d_out + 3) / 4), dim3(256), 0, s, W, mask, d_in, d_out, g, go,
                     capacity, rowptr, Wp, chunk, scale);
  return hipGetLastError();
}

}  // namespace gm
