// The bf16 MFMA GEMM machinery shared by the masked-linear GEMMs and the LM
// head of the distillation loss: XCD-aware tile order, fragment loads, the
// MFMA issue with accumulators tied in place, and the pipelined K-loop over
// LDS stages filled by buffer loads with the lds modifier (gm_pipe.h).
#pragma once

#include <type_traits>

#include "gm_pipe.h"

namespace gm {

// Blocks are dealt to the eight XCDs round-robin; renumber them so that each
// XCD works on a contiguous range of tile indices, then walk the tile grid in
// groups of kGroupM tile rows (column-major inside a group): an XCD's range is
// then a kGroupM-row rectangle of tiles, which shares both operand panels in
// its L2 instead of streaming every panel of one operand.  Eight rows (an
// 8 x 4 rectangle of 256 x 256 tiles per XCD on a 4096 x 4096 output) measured
// 1-3 % faster than four, two or sixteen across the workloads' GEMMs.
constexpr int kGroupM = 8;

__device__ __forceinline__ int xcd_remap(int bid, int nblocks) {
  const int per = nblocks / 8;
  if (per == 0 || bid >= per * 8) return bid;
  return (bid % 8) * per + bid / 8;
}

__device__ __forceinline__ void tile_coords(int bid, int nblocks, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int t = xcd_remap(bid, nblocks);
  const int group = t / (kGroupM * tiles_n);
  const int first_m = group * kGroupM;
  const int gm = min(tiles_m - first_m, kGroupM);
  const int r = t - group * kGroupM * tiles_n;
  tm = first_m + r % gm;
  tn = r / gm;
}

__device__ __forceinline__ void tile_coords(int nblocks, int tiles_m, int tiles_n, int& tm, int& tn) {
  tile_coords(int(blockIdx.x), nblocks, tiles_m, tiles_n, tm, tn);
}

// Accumulator rows mb < kAgprRows<MB> live in AGPRs, the others in arch VGPRs.
template <int MB>
constexpr int kAgprRows = MB - (MB + 3) / 4;

template <int NB, bool KM, int C>
__device__ __forceinline__ void load_bfrags(const u32x4* __restrict__ Bs, int b0, int lane, u32x4 (&bf)[NB]) {
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) bf[nb] = KM ? km_frag(Bs, b0 + nb * 16, lane) : mn_frag<C>(Bs, b0 + nb * 16, lane);
}

template <bool KM, int C>
__device__ __forceinline__ u32x4 load_afrag(const u32x4* __restrict__ As, int a0, int lane) {
  return KM ? km_frag(As, a0, lane) : mn_frag<C>(As, a0, lane);
}

// One MFMA of accumulator (mb, nb); FIRST starts it from zero.
template <bool FIRST, int MB, int NB>
__device__ __forceinline__ void mfma_at(int mb, int nb, const u32x4& af, const u32x4& b, f32x4 (&acc)[MB][NB]) {
  if (mb < kAgprRows<MB>) {
    if constexpr (FIRST) mfma_init<true>(acc[mb][nb], af, b); else mfma_acc<true>(acc[mb][nb], af, b);
  } else {
    if constexpr (FIRST) mfma_init<false>(acc[mb][nb], af, b); else mfma_acc<false>(acc[mb][nb], af, b);
  }
}

template <bool FIRST, int MB, int NB>
__device__ __forceinline__ void mfma_row(int mb, const u32x4& af, const u32x4 (&bf)[NB], f32x4 (&acc)[MB][NB]) {
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) mfma_at<FIRST>(mb, nb, af, bf[nb], acc);
}

// Every fragment row of the wave computes every slice.
struct AllRows {
  __device__ uint32_t operator()(int) const { return ~0u; }
};

// The K-loop shared by the three GEMMs.  `prepare(st)` computes whatever the
// copies of K slice st need (buffer resources, per-lane offsets); it is called
// once per slice, in increasing st, at a point where this wave has no LDS read
// in flight, so any LDS or scalar loads it makes cost only their own latency.
// `issue(st, p)` then starts copy p (0 <= p < PER_STAGE) of slice st into LDS
// buffer st % STAGES; slices st >= nst are never consumed, so their copies
// only need to stay inside their buffer resources.  `landed(st)` runs after
// this wave's copies of slice st completed and before the barrier that
// publishes them (soft-selector rescaling).  `bhook(kt, bf)` sees the B
// fragments of slice kt once they are in registers.  The accumulators are
// written by the first slice's MFMAs (zero when nst is 0).  `live(kt)`
// (wave-uniform) has bit mb set when fragment row mb needs the MFMAs of slice
// kt; rows whose A operand is all zeros for the slice skip them.  The first
// slice runs every row, since its MFMAs also initialise the accumulators.
// XTRA: further DMA instructions per slice that `prepare(st)` itself issues
// (before the slice's copies); the wait counts include them.
//
// Software pipeline: rows 0 .. MB-RA-1 of slice kt run first (A fragments
// streamed one row ahead), and the A fragments of the last RA rows are read;
// then the wave waits for slice kt+1, meets the others at the barrier (which
// also frees buffer kt % STAGES), and issues the last RA MFMA rows of slice kt
// column by column, interleaved with the copies of slice kt + STAGES and the
// reads of slice kt+1's B fragments into the registers those MFMAs have just
// consumed.  Copies run STAGES slices ahead; fragment-read latency and copy
// issue hide behind MFMA work.  RA (rows after the barrier; 1 <= RA <= MB)
// trades MFMAs that cover the barrier wait against MFMAs that cover the next
// slice's B-fragment reads: with MB = 8, four rows after the barrier measured
// 2.5-5 % faster than one for the forward and dgate (six or eight: slower),
// level for dX.  The MFMAs of each accumulator keep their order, so RA does
// not change any result.  Every iteration issues exactly PER_STAGE copies
// (slices past the end copy zeros), so the wait count is a constant, and the
// loop body has no branches around the accumulators; the first and the last
// slice are peeled off.
template <int MB, int NB, bool A_KM, bool B_KM, int CA, int CB, int PER_STAGE, int STAGES, int RA, int XTRA = 0,
          int ABUF, int BBUF, class Prepare, class Issue, class Landed, class BHook, class Live = AllRows>
__device__ __forceinline__ void gemm_mainloop(u32x4 (*As)[ABUF], u32x4 (*Bs)[BBUF], int nst, int a0, int b0, int lane,
                                              f32x4 (&acc)[MB][NB], Prepare&& prepare, Issue&& issue,
                                              Landed&& landed, BHook&& bhook, Live live = Live{}) {
  static_assert(PER_STAGE <= NB, "copies are interleaved with the NB MFMAs of one row");
  static_assert(RA >= 1 && RA <= MB, "rows after the barrier");
  // loads issued after the copies of the slice being waited for: the later
  // slices' copies and the XTRA loads of every prepare() since
  constexpr int AHEAD = (PER_STAGE + XTRA) * (STAGES - 2) + XTRA;
  if (nst <= 0) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    return;
  }
  for (int s = 0; s < STAGES - 1; ++s) {
    prepare(s);
#pragma unroll
    for (int p = 0; p < PER_STAGE; ++p) issue(s, p);
  }
  prepare(STAGES - 1);
  wait_vmcnt<AHEAD>();
  landed(0);
  block_sync();
#pragma unroll
  for (int p = 0; p < PER_STAGE; ++p) issue(STAGES - 1, p);

  u32x4 bf[NB];
  u32x4 af;
  load_bfrags<NB, B_KM, CB>(Bs[0], b0, lane, bf);
  af = load_afrag<A_KM, CA>(As[0], a0, lane);

  // One slice that is followed by another: rows 0 .. MB-RA-1, the barrier,
  // then the last RA rows interleaved with the next slice's copies and
  // fragment reads.
  auto slice = [&](int kt, auto first) {
    constexpr bool FIRST = decltype(first)::value;
    const uint32_t lv = FIRST ? ~0u : live(kt);
    bhook(kt, bf);
    const u32x4* A = As[kt % STAGES];
#pragma unroll
    for (int mb = 0; mb < MB - RA; ++mb) {
      const u32x4 an = load_afrag<A_KM, CA>(A, a0 + (mb + 1) * 16, lane);
      if ((lv >> mb) & 1u) mfma_row<FIRST, MB, NB>(mb, af, bf, acc);
      af = an;
    }
    u32x4 ar[RA];  // A fragments of the rows after the barrier
    ar[0] = af;
#pragma unroll
    for (int r = 1; r < RA; ++r) ar[r] = load_afrag<A_KM, CA>(A, a0 + (MB - RA + r) * 16, lane);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this wave's reads of slice kt are done
    prepare(kt + STAGES);
    wait_vmcnt<AHEAD>();                                 // ... and its copies of slice kt+1
    landed(kt + 1);
    block_sync();
    const u32x4* Bn = Bs[(kt + 1) % STAGES];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
      for (int r = 0; r < RA; ++r)
        if ((lv >> (MB - RA + r)) & 1u) mfma_at<FIRST, MB, NB>(MB - RA + r, nb, ar[r], bf[nb], acc);
      __builtin_amdgcn_sched_barrier(0);
      if (nb < PER_STAGE) issue(kt + STAGES, nb);
      bf[nb] = B_KM ? km_frag(Bn, b0 + nb * 16, lane) : mn_frag<CB>(Bn, b0 + nb * 16, lane);
      __builtin_amdgcn_sched_barrier(0);
    }
    af = load_afrag<A_KM, CA>(As[(kt + 1) % STAGES], a0, lane);
  };
  // The last slice: all rows, no further copies.
  auto last = [&](auto first) {
    constexpr bool FIRST = decltype(first)::value;
    const uint32_t lv = FIRST ? ~0u : live(nst - 1);
    bhook(nst - 1, bf);
    const u32x4* A = As[(nst - 1) % STAGES];
#pragma unroll
    for (int mb = 0; mb < MB - 1; ++mb) {
      const u32x4 an = load_afrag<A_KM, CA>(A, a0 + (mb + 1) * 16, lane);
      if ((lv >> mb) & 1u) mfma_row<FIRST, MB, NB>(mb, af, bf, acc);
      af = an;
    }
    if ((lv >> (MB - 1)) & 1u) mfma_row<FIRST, MB, NB>(MB - 1, af, bf, acc);
  };

  if (nst == 1) {
    last(std::true_type{});
  } else {
    slice(0, std::true_type{});
    for (int kt = 1; kt + 1 < nst; ++kt) slice(kt, std::false_type{});
    last(std::false_type{});
  }
  wait_vmcnt<0>();  // zero-fill copies of slices past the end, before the block exits
  acc_drain<kAgprRows<MB> * NB>(reinterpret_cast<f32x4(&)[MB * NB]>(acc));
}

// Epilogue of a K-loop tile of BM (m) x 256 (n) accumulators, waves 2 (m) x
// NW/2 (n): out[r0 + n][c0 + m] = bf16(C[m][n]) for r0 + n < rlim (c0 + BM <=
// clim or whole 8-column chunks below clim).  The bf16 tile goes through LDS
// as 256 rows of 2 BM bytes (rows 0-127 at lo and 128-255 at hi when BM = 256,
// all at lo otherwise; 16-byte chunk c of row n at slot c ^ (n mod BM/8), so
// the 16 rows of a fragment write different banks), then out as whole rows,
// 16 bytes per lane, nontemporal: full lines that leave no dirty L2 lines for
// the end of the kernel to write back (against 8-byte stores straight from the
// fragments: 2.4 % off the LLaMA-2-7B step, bit-identical).  The first
// barrier waits for every wave's K-loop (its reads and copies are done).
template <int BM, int MB, int NB, int NW>
__device__ __forceinline__ void store_tile_rows(const f32x4 (&acc)[MB][NB], char* lo, char* hi, int wm, int wn,
                                                int tid, int lane, uint16_t* __restrict__ out, int64_t ld, int r0,
                                                int rlim, int c0, int clim) {
  constexpr int CPR = BM / 8;                     // 16-byte chunks per row
  constexpr int RPB = BM == 256 ? 128 : 256;      // rows per LDS buffer
  static_assert(MB * 32 == BM && NB * 16 * (NW / 2) == 256, "tile shape");
  auto row_base = [&](int n) { return (n < RPB ? lo : hi) + (n % RPB) * (2 * BM); };
  __syncthreads();
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int m = wm * (BM / 2) + mb * 16 + 4 * (lane >> 4);
      const int n = wn * NB * 16 + nb * 16 + (lane & 15);
      uint2 w;
      w.x = pack_bf16x2(acc[mb][nb][0], acc[mb][nb][1]);
      w.y = pack_bf16x2(acc[mb][nb][2], acc[mb][nb][3]);
      *reinterpret_cast<uint2*>(row_base(n) + (((m >> 3) ^ (n & (CPR - 1))) << 4) + ((m >> 2) & 1) * 8) = w;
    }
  __syncthreads();
#pragma unroll 4
  for (int k = 0; k < 256 * CPR / (64 * NW); ++k) {
    const int e = k * 64 * NW + tid, n = e / CPR, c = e % CPR;
    const u32x4 v = *reinterpret_cast<const u32x4*>(row_base(n) + ((c ^ (n & (CPR - 1))) << 4));
    if (r0 + n < rlim && c0 + 8 * c < clim)
      __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(out + int64_t(r0 + n) * ld + c0 + 8 * c));
  }
}

}  // namespace gm
