// Column lists of a selector matrix (the group-compacted view of W that the
// dX K-loop walks; Eq. 1): the building unit, shared by the standalone kernel
// and by the dgate launch, whose spare blocks build the lists while its last
// tiles finish.
#pragma once

#include "gm_device.h"

namespace gm {

constexpr int kListChunk = 1024;  // rows per unit

// Unit `unit` = (list column c, chunk k of 1024 rows) on a block of NT threads
// (NT = 512 or 1024, 1024 / NT rows per thread).  The unit counts the kept rows
// of chunks 0 .. k-1 itself (every thread loads its share of those selectors
// and of its own rows at once: one memory round trip), then places its chunk's
// kept rows after them in increasing order with block-wide exclusive scans (a
// shuffle scan inside each wave, then the wave totals in LDS), one per NT-row
// part of the chunk.  The unit of the last chunk writes the column's count and
// soft flag.  Every thread of the block must call it (it has barriers).
template <int NT>
__device__ __forceinline__ void col_lists_unit(int unit, int nchunks, const float* __restrict__ mask, int d_out,
                                               int G_in, int go, int nsub, int* __restrict__ colcount,
                                               int* __restrict__ colsoft, int* __restrict__ rows,
                                               float* __restrict__ scales, int* __restrict__ subbits) {
  static_assert(NT == 512 || NT == 1024, "block size");
  constexpr int R = kListChunk / NT, NWV = NT / 64;
  __shared__ int s_tot[NWV];
  __shared__ int s_red[NWV];
  const int c = unit / nchunks, k = unit % nchunks;
  const int tid = int(threadIdx.x), lane = tid & 63, w = tid >> 6;
  auto kept_bits = [&](int o, float(&m)[4]) {
    int b = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      m[q] = (q < nsub && o < d_out) ? mask[int64_t(o / go) * G_in + c * nsub + q] : 0.0f;
      b |= int(m[q] != 0.0f) << q;
    }
    return b;
  };
  auto block_sum = [&](int v) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d);
    if (lane == 0) s_red[w] = v;
    __syncthreads();
    int t = 0;
#pragma unroll
    for (int q = 0; q < NWV; ++q) t += s_red[q];
    __syncthreads();
    return t;
  };
  // this thread's rows of the chunk, and its rows of the preceding chunks
  float m[R][4];
  int bits[R];
#pragma unroll
  for (int r = 0; r < R; ++r) bits[r] = kept_bits(k * kListChunk + r * NT + tid, m[r]);
  bool soft = false;
  int before = 0;
  for (int kk = 0; kk < k; ++kk)
#pragma unroll
    for (int r = 0; r < R; ++r) {
      float mp[4];
      before += kept_bits(kk * kListChunk + r * NT + tid, mp) != 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) soft |= mp[q] != 0.0f && mp[q] != 1.0f;
    }
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int q = 0; q < 4; ++q) soft |= m[r][q] != 0.0f && m[r][q] != 1.0f;
  int off = block_sum(before);  // kept rows before this part of the chunk
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int cnt = bits[r] != 0;
    int inc = cnt;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int up = __shfl_up(inc, d);
      if (lane >= d) inc += up;
    }
    if (lane == 63) s_tot[w] = inc;
    __syncthreads();
    int pre = 0, tot = 0;
#pragma unroll
    for (int q = 0; q < NWV; ++q) {
      const int t = s_tot[q];
      if (q < w) pre += t;
      tot += t;
    }
    if (bits[r]) {
      const int64_t e = int64_t(c) * d_out + off + pre + inc - cnt;
      rows[e] = k * kListChunk + r * NT + tid;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (q < nsub) scales[e * nsub + q] = m[r][q];
      if (nsub > 1) subbits[e] = bits[r];
    }
    off += tot;
    __syncthreads();  // s_tot is read before the next part overwrites it
  }
  if (k == nchunks - 1) {
    const int any_soft = block_sum(int(soft));
    if (tid == 0) {
      colcount[c] = off;
      colsoft[c] = any_soft != 0;
    }
  }
}

}  // namespace gm
