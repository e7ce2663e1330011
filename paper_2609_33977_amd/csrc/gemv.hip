// Decode-sized forward of a group-masked linear: Y[t, o] = sum over the kept
// groups (o / g_out, v) of mask[o / g_out, v] * sum_{i in v} X[t, i] W[o, i],
// for up to 16 tokens per pass (Eq. 1 applied to the pruned model's linear).
//
// One wave per output row.  The row's part of a group, g bf16 weights, is g*2 contiguous bytes;
// the wave covers 512 consecutive weights per step (512/g groups side by side,
// 16 bytes per lane), so every kept weight is read from HBM exactly once per
// pass and pruned groups are never touched.  Bytes per pass: 2 * nnz (kept
// weights) + index/mask + 2 T (d_in + d_out); the kernel is HBM-bound for small T.
//
// Two layouts of the same row-major kept-group sequence:
//   in place : W [d_out, d_in] with the mask deciding which groups are read;
//   packed   : Wp [k, g] + chunk [k] + scale [k] + rowptr [d_out + 1] written
//              by the export (Appendix F), the row's groups contiguous.
#include "gm_device.h"
#include "gm_launch.h"
#include "gm_pipe.h"

namespace gm {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Dot product of two vectors of 8 bf16 with fp32 accumulation (v_dot2_f32_bf16).
// The bf16 pairs are moved out of the 32-bit lanes with memcpy: a bit_cast of
// a subscripted vector element inside this unrolled loop was folded to element
// 0 by the compiler (every step used the first pair).
__device__ __forceinline__ float dot8_bf16(u32x4 w, u32x4 x) {
  const uint32_t wa[4] = {w.x, w.y, w.z, w.w};
  const uint32_t xa[4] = {x.x, x.y, x.z, x.w};
  float acc = 0.0f;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    bf16x2 a, b;
    __builtin_memcpy(&a, &wa[q], sizeof(a));
    __builtin_memcpy(&b, &xa[q], sizeof(b));
    acc = __builtin_amdgcn_fdot2_f32_bf16(a, b, acc, false);
  }
  return acc;
}

constexpr int kMaxGroupsPerRow = 1024;  // G_in limit of the in-place variant's per-wave list

// MAXG: capacity of the in-place variant's per-wave list (512 or 1024; the
// smaller list leaves more LDS for other blocks).  A row reads mask row o / go.
template <int TB, bool PACKED, int MAXG>
__global__ __launch_bounds__(256) void gemv_kernel(const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
                                                   const float* __restrict__ mask,
                                                   const uint16_t* __restrict__ Wp, const int* __restrict__ chunk,
                                                   const float* __restrict__ scale,
                                                   const int* __restrict__ rowptr, int T, int t0, int d_in,
                                                   int d_out, int g, int go, uint16_t* __restrict__ Y) {
  __shared__ int s_v[4][PACKED ? 1 : MAXG];
  __shared__ float s_m[4][PACKED ? 1 : MAXG];
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const int o = blockIdx.x * 4 + wv;
  if (o >= d_out) return;  // whole wave leaves together; no block barrier below
  const int G_in = d_in / g;
  const int lanes_per_group = g >> 3;
  const int gps = 64 / lanes_per_group;  // groups per wave step (>= 1 for g <= 512)
  const int slot = lane / lanes_per_group;
  const int e = (lane % lanes_per_group) * 8;
  const int ntok = min(TB, T - t0);

  int nk;
  int64_t pbase = 0;
  if constexpr (PACKED) {
    pbase = rowptr[o];
    nk = rowptr[o + 1] - int(pbase);
  } else {
    // Compact this row's kept groups into the wave's LDS list, in column order.
    nk = 0;
    for (int vb = 0; vb < G_in; vb += 64) {
      const int v = vb + lane;
      const float m = v < G_in ? mask[int64_t(o / go) * G_in + v] : 0.0f;
      const uint64_t bal = __ballot(m != 0.0f);
      if (m != 0.0f) {
        const int r = nk + __popcll(bal & ((uint64_t(1) << lane) - 1));
        s_v[wv][r] = v;
        s_m[wv][r] = m;
      }
      nk += __popcll(bal);
    }
    // LDS writes of this wave become visible to its other lanes before the list is read.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }

  float acc[TB];
#pragma unroll
  for (int t = 0; t < TB; ++t) acc[t] = 0.0f;

  for (int k0 = 0; k0 < nk; k0 += 2 * gps) {
    const int ka = k0 + slot;
    const int kb = k0 + gps + slot;
    int va = 0, vb = 0;
    float ma = 0.0f, mb = 0.0f;
    u32x4 wa = zero16(), wb = zero16();
    if (ka < nk) {
      if constexpr (PACKED) {
        va = chunk[pbase + ka];
        ma = scale[pbase + ka];
        wa = ld16(Wp + (pbase + ka) * g + e);
      } else {
        va = s_v[wv][ka];
        ma = s_m[wv][ka];
        wa = ld16(W + int64_t(o) * d_in + int64_t(va) * g + e);
      }
    }
    if (kb < nk) {
      if constexpr (PACKED) {
        vb = chunk[pbase + kb];
        mb = scale[pbase + kb];
        wb = ld16(Wp + (pbase + kb) * g + e);
      } else {
        vb = s_v[wv][kb];
        mb = s_m[wv][kb];
        wb = ld16(W + int64_t(o) * d_in + int64_t(vb) * g + e);
      }
    }
#pragma unroll
    for (int t = 0; t < TB; ++t) {
      if (t < ntok) {
        const uint16_t* xr = X + int64_t(t0 + t) * d_in + e;
        float p = 0.0f;
        if (ka < nk) p += ma * dot8_bf16(wa, ld16(xr + int64_t(va) * g));
        if (kb < nk) p += mb * dot8_bf16(wb, ld16(xr + int64_t(vb) * g));
        acc[t] += p;
      }
    }
  }

#pragma unroll
  for (int t = 0; t < TB; ++t) {
    float s = acc[t];
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) s += __shfl_xor(s, d);
    acc[t] = s;
  }
  if (lane == 0) {
#pragma unroll
    for (int t = 0; t < TB; ++t)
      if (t < ntok) Y[int64_t(t0 + t) * d_out + o] = uint16_t(f32_to_bf16_bits(acc[t]));
  }
}

// 16 bytes through a buffer resource; an offset past the resource's range
// reads zeros.  cpol: cache policy bits (kCpolNt: nontemporal).
constexpr uint32_t kOutOfRange = 0x80000000u;
constexpr int kCpolNt = 2;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t t1_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), short(0), int(bytes), 0x00020000);
}

__device__ __forceinline__ u32x4 ld16_rsrc(__amdgpu_buffer_rsrc_t r, uint32_t off, int cpol) {
  return cpol == kCpolNt ? __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kCpolNt))
                         : __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// ---------------------------------------------------------------- 2..16 tokens

// For a batch of 2..16 tokens the one-wave-per-row kernel re-reads X for
// every row.  This variant computes 16 RT output rows per block with
// v_mfma_f32_16x16x32_bf16 (M = rows, N = tokens padded to 16, K = 32 input
// columns per instruction): a 16-byte chunk of X feeds the RT row tiles of 16
// rows, so X is read from L2 once per 16 RT rows instead of once per row.  The
// eight waves of the block split the input columns and sum their partial tiles
// in LDS in wave order.  The mask rows of the block are staged in LDS first; a
// lane reads a W chunk only when its group is kept (pruned chunks are zeros),
// so HBM traffic is the kept weights, as in the GEMV.  The packed export runs
// the same K loop: the block turns its rows' piece lists into the same
// (row, group) table, with each kept group's piece index beside its selector,
// and reads the pieces instead of W's rows; both layouts therefore give
// identical results.  The weights go through the caches: an instruction
// reads 64 bytes of each of 16 rows, and the other half of each 128-byte line
// is requested by the very next instruction (nontemporal loads measured 3-8 %
// slower here).  In the MFMA operand layout adjacent lanes hold different
// rows, so every active lane of such a load was a cache access of its own
// (32 per instruction at half the groups kept); the weights are therefore
// loaded with four adjacent lanes per 64-byte row segment (one access per
// kept row) and moved into the operand layout with ds_bpermute: 4-10 %
// faster on the LLaMA-2-13B shapes at 2-16 tokens, identical results.
// X has the same problem (one access per active lane).  Permuting it too
// saved 0.5 us at 16 tokens and cost as much at 2 and 8; copying each batch's
// X slices into LDS with buffer loads (four lanes per token segment) and
// reading the operands from there is 2-4 % faster for blocks of 64 rows at
// every token count and for 32-row blocks at 16 tokens (2-5 %), but 2-4 %
// slower for 32-row blocks at 2 and 8 tokens, which keep the direct loads.
constexpr int kMmaWaves = 8;
constexpr int kMmaMaskFloats = 8192;  // staged mask floats per block: mask rows of the block x selectors per row

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// XL: X goes through LDS (see the K loop); the launcher picks it for blocks of
// 64 rows, or more than 8 tokens, where it measured 2-5 % faster.
template <int RT, bool PACKED, bool XL>
__global__ __launch_bounds__(64 * kMmaWaves) void gemv_mfma_kernel(const uint16_t* __restrict__ X,
                                                                  const uint16_t* __restrict__ W,
                                                                  const float* __restrict__ mask,
                                                                  const int* __restrict__ chunk,
                                                                  const float* __restrict__ scale,
                                                                  const int* __restrict__ rowptr, int T, int d_in,
                                                                  int d_out, int g, int go,
                                                                  uint16_t* __restrict__ Y) {
  constexpr int R = 16 * RT;
  constexpr int NT = 64 * kMmaWaves;
  __shared__ float s_m[kMmaMaskFloats];
  __shared__ int s_idx[PACKED ? kMmaMaskFloats : 1];  // packed: piece of (row, group) from the block's first piece
  __shared__ int s_rp[PACKED ? R + 1 : 1];
  __shared__ f32x4 s_part[kMmaWaves][RT][64];
  __shared__ u32x4 s_x[kMmaWaves][XL ? 4 * 64 : 1];  // XL: per wave, the X slices of one load batch
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int o0 = blockIdx.x * R;
  const int G_in = d_in / g;
  const int mrows = go == 1 ? R : (R > go ? R / go : 1);
  const int u0 = o0 / go;
  const int G_out = (d_out + go - 1) / go;
  const int rows = min(R, d_out - o0);  // rows of this block inside W
  // Staged selectors; the block notes whether any lies strictly between 0 and
  // 1 (a soft selector), so that the K loop scales weights only in blocks
  // that hold one and carries no per-slice branch otherwise.  In place the
  // selectors are the mask rows of the block.  Packed (W = Wp, go = 1), the
  // table starts at zero (pruned) and every piece p of the block's rows
  // writes its selector scale[p] and its index into (row, chunk[p]); pieces
  // whose column is out of range are ignored.
  int soft_here = 0;
  int p0 = 0;  // packed: first piece of the block
  if constexpr (PACKED) {
    for (int e = tid; e <= rows; e += NT) s_rp[e] = rowptr[o0 + e];
    for (int e = tid; e < R * G_in; e += NT) s_m[e] = 0.0f;
    __syncthreads();
    p0 = s_rp[0];
    const int np = s_rp[rows] - p0;
    for (int e = tid; e < np; e += NT) {
      int lo = 0, hi = rows;  // the row of piece p0 + e: s_rp[lo] <= p0 + e < s_rp[lo + 1]
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (s_rp[mid] <= p0 + e) lo = mid; else hi = mid;
      }
      const int v = chunk[p0 + e];
      if (v >= 0 && v < G_in) {
        const float sv = scale[p0 + e];
        s_m[lo * G_in + v] = sv;
        s_idx[lo * G_in + v] = e;
        soft_here |= sv != 0.0f && sv != 1.0f;
      }
    }
  } else {
    for (int e = tid; e < mrows * G_in; e += NT) {
      const int rr = e / G_in;
      const float v = u0 + rr < G_out ? mask[int64_t(u0) * G_in + e] : 0.0f;
      s_m[e] = v;
      soft_here |= v != 0.0f && v != 1.0f;
    }
  }
  const bool soft = __syncthreads_or(soft_here);

  const int r = lane & 15, kc = lane >> 4;
  // W is loaded with four adjacent lanes per 64-byte row segment (row rl,
  // 16-byte chunk cl) and moved into the MFMA operand layout (row r, chunk kc)
  // by a lane permutation: lane l takes the data of lane 4 (l & 15) + (l >> 4).
  const int rl = lane >> 2, cl = lane & 3;
  const int bpa = (4 * r + kc) * 4;
  const float* mrow[RT];
  uint32_t wrow[RT];  // byte offset of this lane's row (and 16-byte column chunk) in W
  bool orow[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    const int o = o0 + rt * 16 + rl;
    orow[rt] = o < d_out;
    mrow[rt] = s_m + (go == 1 ? rt * 16 + rl : (o0 + rt * 16) / go - u0) * G_in;
    wrow[rt] = (uint32_t(rt * 16 + rl) * uint32_t(d_in) + uint32_t(8 * cl)) * 2u;
  }
  const bool tok = r < T;
  const uint32_t xrow = (uint32_t(tok ? r : 0) * uint32_t(d_in) + uint32_t(8 * kc)) * 2u;
  // XL: four adjacent lanes copy one token's 64-byte segment of a slice into
  // LDS (lane 4 t + j takes chunk j ^ ((t >> 2) & 3), so that the operand
  // reads, chunk kc of token r, hit distinct banks): one cache access per
  // token instead of one per lane.
  const int xt = lane >> 2;
  const bool xtok = xt < T;
  const uint32_t xoff = (uint32_t(xtok ? xt : 0) * uint32_t(d_in) + uint32_t(8 * ((lane & 3) ^ ((xt >> 2) & 3)))) * 2u;
  const i32x4_t rxd = make_rsrc_grouped(X, uint32_t(T) * uint32_t(d_in) * 2u);
  const uint32_t xlds = XL ? lds_addr(&s_x[wave][0]) : 0u;
  const int xread = r * 4 + ((kc ^ (r >> 2)) & 3);  // this lane's operand chunk in a slice of s_x
  // the block's rows of W (packed: the block's pieces) and the T rows of X
  // (the launcher keeps both under 2 GiB)
  const __amdgpu_buffer_rsrc_t rw =
      PACKED ? t1_rsrc(W + int64_t(p0) * g, uint32_t(s_rp[rows] - p0) * uint32_t(g) * 2u)
             : t1_rsrc(W + int64_t(o0) * d_in, uint32_t(rows * d_in) * 2u);
  const __amdgpu_buffer_rsrc_t rx = t1_rsrc(X, uint32_t(T) * uint32_t(d_in) * 2u);
  const int lg = __builtin_ctz(unsigned(g));  // g is a power of two: the group of a column by shift
  const int nsl = d_in / 32;
  const int s0 = wave * nsl / kMmaWaves, s1 = (wave + 1) * nsl / kMmaWaves;
  f32x4 acc[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) acc[rt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  constexpr int U = 4;  // K slices of 32 columns per load batch
  // Batches of U slices.  The selectors of batch b + 1 are read from LDS while
  // batch b's loads are in flight, so no LDS round trip sits between a batch's
  // loads; the loads themselves are branch-free buffer loads (a pruned group,
  // a slice past the wave's range, a row past d_out or a token past T reads
  // zeros through an out-of-range offset, without a memory access).
  float mn[RT][U];
  uint32_t on[RT][U];  // packed: byte offset of the lane's 16 bytes in the block's pieces
  auto read_masks = [&](int sb) {
#pragma unroll
    for (int q = 0; q < U; ++q) {
      const int k = (sb + q) * 32;
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int at = int(mrow[rt] - s_m) + ((k + 8 * cl) >> lg);
        mn[rt][q] = sb + q < s1 && orow[rt] ? s_m[at] : 0.0f;
        if constexpr (PACKED)
          on[rt][q] = sb + q < s1 && orow[rt]
                          ? (uint32_t(s_idx[at]) * uint32_t(g) + uint32_t((k + 8 * cl) & (g - 1))) * 2u
                          : kOutOfRange;
      }
    }
  };
  auto k_loop = [&](auto soft_tag) {
    read_masks(s0);
    for (int sb = s0; sb < s1; sb += U) {
      float m[RT][U];
      u32x4 av[RT][U], bv[U];
      if constexpr (XL) {  // before the weight loads, so that the wait below counts those after them
        static_assert(U == 4, "one grouped copy per slice of the batch");
        dma16_group<0>(rxd, group_voffset(sb + 0 < s1 && xtok ? xoff + uint32_t(sb + 0) * 64u : kOOB, 0), xlds);
        dma16_group<1>(rxd, group_voffset(sb + 1 < s1 && xtok ? xoff + uint32_t(sb + 1) * 64u : kOOB, 1), xlds);
        dma16_group<2>(rxd, group_voffset(sb + 2 < s1 && xtok ? xoff + uint32_t(sb + 2) * 64u : kOOB, 2), xlds);
        dma16_group<3>(rxd, group_voffset(sb + 3 < s1 && xtok ? xoff + uint32_t(sb + 3) * 64u : kOOB, 3), xlds);
      }
      // Row tile by row tile, consecutive slices back to back: the two 64-byte
      // halves of a row's 128-byte line (slices 2j and 2j + 1) are requested by
      // adjacent instructions (measured 15-25 % faster on 13824 x 5120 than
      // slice-major order, which spaces the halves RT instructions apart).
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int q = 0; q < U; ++q) {
          m[rt][q] = mn[rt][q];
          const uint32_t off = PACKED ? on[rt][q] : wrow[rt] + uint32_t(sb + q) * 64u;
          av[rt][q] = ld16_rsrc(rw, m[rt][q] != 0.0f ? off : kOutOfRange, 0);
        }
      if constexpr (XL) {
        read_masks(sb + U);
        wait_vmcnt<RT * U>();  // the X copies (issued before the RT U weight loads) have landed
#pragma unroll
        for (int q = 0; q < U; ++q) bv[q] = s_x[wave][q * 64 + xread];
      } else {
#pragma unroll
        for (int q = 0; q < U; ++q)
          bv[q] = ld16_rsrc(rx, sb + q < s1 && tok ? xrow + uint32_t(sb + q) * 64u : kOutOfRange, 0);
        read_masks(sb + U);
      }
#pragma unroll
      for (int q = 0; q < U; ++q)
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          const float mq = m[rt][q];
          u32x4 aq = av[rt][q];
          if constexpr (decltype(soft_tag)::value) aq = scale_bf16x8(aq, mq);
          aq = u32x4{uint32_t(__builtin_amdgcn_ds_bpermute(bpa, int(aq.x))),
                     uint32_t(__builtin_amdgcn_ds_bpermute(bpa, int(aq.y))),
                     uint32_t(__builtin_amdgcn_ds_bpermute(bpa, int(aq.z))),
                     uint32_t(__builtin_amdgcn_ds_bpermute(bpa, int(aq.w)))};
          acc[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, aq),
                                                            __builtin_bit_cast(bf16x8, bv[q]), acc[rt], 0, 0, 0);
        }
    }
  };
  if (soft)
    k_loop(std::true_type{});
  else
    k_loop(std::false_type{});
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) s_part[wave][rt][lane] = acc[rt];
  __syncthreads();
  if (wave < RT) {
    const int rt = wave;
    f32x4 sum = s_part[0][rt][lane];
#pragma unroll
    for (int w = 1; w < kMmaWaves; ++w) sum += s_part[w][rt][lane];
    const int ob = o0 + rt * 16 + 4 * kc;
    if (r < T && ob < d_out) {
      uint2 v;
      v.x = pack_bf16x2(sum[0], sum[1]);
      v.y = pack_bf16x2(sum[2], sum[3]);
      *reinterpret_cast<uint2*>(Y + int64_t(r) * d_out + ob) = v;
    }
  }
}

// ---------------------------------------------------------------- one token

// One token: one wave per output row.  The lane's groups of the row are the
// kept groups with index k = slot, slot + gps, slot + 2 gps, ... in column
// order, and the weight loads of up to kT1Steps such steps (16 bytes per lane
// each) are issued together.  Four steps keep the kernel at 62 registers, so
// eight waves per SIMD are resident: on the LLaMA-2-13B projections that
// streams 8 % faster than eight steps per chunk at four waves per SIMD (more
// rows in flight beats more loads per row).  In place (rows of at most 64
// groups), the lanes read the row's selectors at once and compact the kept
// ones into a per-wave LDS list (column, selector) by rank; the weight and
// input loads of a step then go out together.  Packed, the row's pieces are
// contiguous from rowptr[o] with their column in chunk[] and selector in
// scale[]: the piece addresses need only the row pointer, so a chunk's weight
// loads are issued before its (column, selector) list arrives, through buffer
// loads whose out-of-range offsets read zeros (no branches, so the compiler
// can wait for the list without waiting for the weights).  Weights are
// streamed once, so they are loaded nontemporal (they would only evict the
// input vector and the selectors from the caches); X is read through the
// caches (every row reuses it).  Both layouts accumulate the same products in
// the same order, and the row sum is a fixed-order 64-lane reduction, so
// their results are identical.
constexpr int kT1Steps = 4;

template <bool PACKED>
__global__ __launch_bounds__(256) void gemv_t1_kernel(const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
                                                      const float* __restrict__ mask,
                                                      const uint16_t* __restrict__ Wp, const int* __restrict__ chunk,
                                                      const float* __restrict__ scale,
                                                      const int* __restrict__ rowptr, int d_in, int d_out, int g,
                                                      int go, uint16_t* __restrict__ Y) {
  __shared__ int s_v[4][PACKED ? 1 : 64];
  __shared__ float s_m[4][PACKED ? 1 : 64];
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform, so the row's resource is too
  const int o = int(blockIdx.x) * 4 + wv;
  if (o >= d_out) return;  // whole wave leaves together; no block barrier below
  const int G_in = d_in / g;  // at most 64 in place
  const int lpg = g >> 3;     // lanes per group (16 bytes each)
  const int gps = 64 / lpg;   // groups per step
  const int slot = lane / lpg;
  const int e = (lane % lpg) * 8;
  // The row's kept groups as a list (column, selector), 64 entries at a time:
  // in place from a ballot over the row's selectors (at most 64, one batch),
  // kept in LDS; packed from chunk[] and scale[] with one coalesced load per
  // batch, kept in registers and read across lanes.
  int nk;
  int64_t pb = 0;
  uint64_t bits = 0;
  float mv = 0.0f;
  if constexpr (PACKED) {
    const int p0 = __builtin_amdgcn_readfirstlane(rowptr[o]);  // the same for every lane
    pb = p0;
    nk = __builtin_amdgcn_readfirstlane(rowptr[o + 1]) - p0;
  } else {
    mv = lane < G_in ? mask[int64_t(o / go) * G_in + lane] : 0.0f;
    bits = __ballot(mv != 0.0f);
    nk = __popcll(bits);
  }
  // Packed: byte ranges of the row's weights and of X (loads at an offset
  // past the range return zeros: dead steps need no branch).
  const uint16_t* wrow = PACKED ? Wp + pb * g : W + int64_t(o) * d_in;  // wave-uniform
  const __amdgpu_buffer_rsrc_t rw = t1_rsrc(wrow, PACKED ? uint32_t(nk * g) * 2u : 0u);
  const __amdgpu_buffer_rsrc_t rx = t1_rsrc(X, PACKED ? uint32_t(d_in) * 2u : 0u);
  float acc = 0.0f;
  for (int kb = 0; kb < nk; kb += 64) {
    // packed: lane j holds entry kb + j of the row's list (one coalesced load);
    // in place: the list goes to LDS by rank
    int cv = 0;
    float cs = 0.0f;
    if constexpr (PACKED) {
      if (kb + lane < nk) {
        cv = chunk[pb + kb + lane];
        cs = scale[pb + kb + lane];
      }
    } else {
      if (mv != 0.0f) {
        const int r = __builtin_amdgcn_mbcnt_hi(uint32_t(bits >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(bits), 0u));
        s_v[wv][r] = lane;
        s_m[wv][r] = mv;
      }
      // LDS writes of this wave become visible to its other lanes before the list is read.
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    const int nb = min(64, nk - kb);
    for (int k0 = 0; k0 < nb; k0 += kT1Steps * gps) {
      u32x4 w[kT1Steps], x[kT1Steps];
      float m[kT1Steps];
      int v[kT1Steps];
      if constexpr (PACKED) {
        // the weights need only the row pointer: issued before the list arrives
        // (branch-free, so the list can be waited for without the weights)
#pragma unroll
        for (int c = 0; c < kT1Steps; ++c) {
          const int kk = k0 + c * gps + slot;
          w[c] = ld16_rsrc(rw, kk < nb ? (uint32_t(kb + kk) * uint32_t(g) + uint32_t(e)) * 2u : kOutOfRange, kCpolNt);
        }
        // every lane takes part in both reads (a lane reads from a lane whose
        // own step may be past the list), then dead steps drop their selector
#pragma unroll
        for (int c = 0; c < kT1Steps; ++c) {
          const int kk = k0 + c * gps + slot;
          const int k = min(kk, 63);
          v[c] = __shfl(cv, k);
          const float ms = __shfl(cs, k);
          m[c] = kk < nb ? ms : 0.0f;
        }
#pragma unroll
        for (int c = 0; c < kT1Steps; ++c)
          x[c] = ld16_rsrc(rx, k0 + c * gps + slot < nb ? uint32_t(v[c] * g + e) * 2u : kOutOfRange, 0);
      } else {
        // in place the weights wait for the list anyway: plain loads, weight and input together
#pragma unroll
        for (int c = 0; c < kT1Steps; ++c) {
          const int k = k0 + c * gps + slot;
          const bool live = k < nb;
          v[c] = 0;
          m[c] = 0.0f;
          w[c] = zero16();
          x[c] = zero16();
          if (live) {
            v[c] = s_v[wv][k];
            m[c] = s_m[wv][k];
            w[c] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wrow + v[c] * g + e));
            x[c] = ld16(X + v[c] * g + e);
          }
        }
      }
#pragma unroll
      for (int c = 0; c < kT1Steps; ++c) acc += m[c] * dot8_bf16(w[c], x[c]);
    }
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) acc += __shfl_xor(acc, d);
  if (lane == 0) Y[o] = uint16_t(f32_to_bf16_bits(acc));
}

template <bool PACKED>
static hipError_t launch_t1(const uint16_t* X, const uint16_t* W, const float* mask, const uint16_t* Wp,
                            const int* chunk, const float* scale, const int* rowptr, int d_in, int d_out, int g,
                            int go, uint16_t* Y, hipStream_t s) {
  hipLaunchKernelGGL(gemv_t1_kernel<PACKED>, dim3(unsigned((d_out + 3) / 4)), dim3(256), 0, s, X, W, mask, Wp, chunk,
                     scale, rowptr, d_in, d_out, g, go, Y);
  return hipGetLastError();
}

template <bool PACKED, int MAXG>
static hipError_t gemv_passes(const uint16_t* X, const uint16_t* W, const float* mask, const uint16_t* Wp,
                              const int* chunk, const float* scale, const int* rowptr, int T, int d_in, int d_out,
                              int g, int go, uint16_t* Y, hipStream_t s) {
  const dim3 grid((d_out + 3) / 4), block(256);
  for (int t0 = 0; t0 < T; t0 += 16) {
    const int nt = T - t0;
    if (nt == 1)
      hipLaunchKernelGGL((gemv_kernel<1, PACKED, MAXG>), grid, block, 0, s, X, W, mask, Wp, chunk, scale, rowptr, T,
                         t0, d_in, d_out, g, go, Y);
    else if (nt <= 4)
      hipLaunchKernelGGL((gemv_kernel<4, PACKED, MAXG>), grid, block, 0, s, X, W, mask, Wp, chunk, scale, rowptr, T,
                         t0, d_in, d_out, g, go, Y);
    else if (nt <= 8)
      hipLaunchKernelGGL((gemv_kernel<8, PACKED, MAXG>), grid, block, 0, s, X, W, mask, Wp, chunk, scale, rowptr, T,
                         t0, d_in, d_out, g, go, Y);
    else
      hipLaunchKernelGGL((gemv_kernel<16, PACKED, MAXG>), grid, block, 0, s, X, W, mask, Wp, chunk, scale, rowptr, T,
                         t0, d_in, d_out, g, go, Y);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// The 2..16 token MFMA kernel when its staged tables fit in LDS and its byte
// offsets fit in 32 bits: four row tiles while that still gives 192 blocks or
// more, else two, fewer when the block's tables do not fit.  Returns false
// (nothing launched) otherwise.
template <bool PACKED>
static bool launch_mfma(const uint16_t* X, const uint16_t* W, const float* mask, const int* chunk, const float* scale,
                        const int* rowptr, int T, int d_in, int d_out, int g, int go, uint16_t* Y, hipStream_t s,
                        hipError_t& err) {
  const int G_in = d_in / g;
  auto fits = [&](int R) { return (go == 1 ? R : (R > go ? R / go : 1)) * G_in <= kMmaMaskFloats; };
  int rt = (d_out + 63) / 64 >= 192 ? 4 : 2;
  while (rt > 1 && !fits(16 * rt)) rt /= 2;
  // byte offsets into the block's rows of W (or its pieces) and into X are 32-bit, below the out-of-range marker
  const int64_t span = int64_t(16 * rt > T ? 16 * rt : T) * d_in * 2;
  if (!fits(16 * rt) || span >= int64_t(kOutOfRange)) return false;
  const dim3 grid(unsigned((d_out + 16 * rt - 1) / (16 * rt))), block(64 * kMmaWaves);
  const bool xl = rt == 4 || T > 8;
#define GM_MFMA_LAUNCH(RTV, XLV)                                                                                  \
  hipLaunchKernelGGL((gemv_mfma_kernel<RTV, PACKED, XLV>), grid, block, 0, s, X, W, mask, chunk, scale, rowptr, T, \
                     d_in, d_out, g, go, Y)
  if (rt == 4) {
    if (xl) GM_MFMA_LAUNCH(4, true); else GM_MFMA_LAUNCH(4, false);
  } else if (rt == 2) {
    if (xl) GM_MFMA_LAUNCH(2, true); else GM_MFMA_LAUNCH(2, false);
  } else {
    if (xl) GM_MFMA_LAUNCH(1, true); else GM_MFMA_LAUNCH(1, false);
  }
#undef GM_MFMA_LAUNCH
  err = hipGetLastError();
  return true;
}

hipError_t launch_gemv_inplace(const uint16_t* X, const uint16_t* W, const float* mask, int T, int d_in, int d_out,
                               int g, int go, uint16_t* Y, hipStream_t s) {
  hipError_t err = hipSuccess;
  if (T >= 2 && T <= 16 && launch_mfma<false>(X, W, mask, nullptr, nullptr, nullptr, T, d_in, d_out, g, go, Y, s, err))
    return err;
  if (T == 1 && d_in / g <= 64)
    return launch_t1<false>(X, W, mask, nullptr, nullptr, nullptr, nullptr, d_in, d_out, g, go, Y, s);
  if (d_in / g <= 512)
    return gemv_passes<false, 512>(X, W, mask, nullptr, nullptr, nullptr, nullptr, T, d_in, d_out, g, go, Y, s);
  return gemv_passes<false, kMaxGroupsPerRow>(X, W, mask, nullptr, nullptr, nullptr, nullptr, T, d_in, d_out, g, go,
                                              Y, s);
}

hipError_t launch_gemv_packed(const uint16_t* X, const uint16_t* Wp, const int* chunk, const float* scale,
                              const int* rowptr, int T, int d_in, int d_out, int g, uint16_t* Y, hipStream_t s) {
  if (T == 1) return launch_t1<true>(X, nullptr, nullptr, Wp, chunk, scale, rowptr, d_in, d_out, g, 1, Y, s);
  hipError_t err = hipSuccess;
  if (T <= 16 && launch_mfma<true>(X, Wp, nullptr, chunk, scale, rowptr, T, d_in, d_out, g, 1, Y, s, err)) return err;
  return gemv_passes<true, 1>(X, nullptr, nullptr, Wp, chunk, scale, rowptr, T, d_in, d_out, g, 1, Y, s);
}

int gemv_max_groups_per_row() { return kMaxGroupsPerRow; }

}  // namespace gm
