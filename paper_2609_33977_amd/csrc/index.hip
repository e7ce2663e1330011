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
#include "gm_lists.h"

namespace gm {

// One 1024-thread block per list column c and chunk of 1024 rows, so that the
// chunks of a column run side by side (col_lists_unit).  Against one block
// per column walking its chunks in turn: 7.8 -> 6.6 us for 4096 rows, 19.4 ->
// 9.2 us for 11008 rows (LLaMA-2-7B shapes, 16 list columns), identical lists.
__global__ __launch_bounds__(1024) void col_lists_kernel(const float* __restrict__ mask, int d_out, int G_in,
                                                        int go, int nsub, int nchunks, int* __restrict__ colcount,
                                                        int* __restrict__ colsoft, int* __restrict__ rows,
                                                        float* __restrict__ scales, int* __restrict__ subbits) {
  col_lists_unit<1024>(int(blockIdx.x), nchunks, mask, d_out, G_in, go, nsub, colcount, colsoft, rows, scales,
                       subbits);
}

hipError_t launch_col_lists(const float* mask, int d_out, int G_in, int go, int nsub, int* colcount, int* colsoft,
                            int* rows, float* scales, int* subbits, hipStream_t s) {
  const int nchunks = (d_out + kListChunk - 1) / kListChunk;
  hipLaunchKernelGGL(col_lists_kernel, dim3((G_in / nsub) * nchunks), dim3(1024), 0, s, mask, d_out, G_in, go, nsub,
                     nchunks, colcount, colsoft, rows, scales, subbits);
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
