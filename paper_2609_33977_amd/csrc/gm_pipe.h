// Building blocks of the pipelined LDS GEMMs on gfx950: asynchronous
// global -> LDS copies, explicit memory-counter waits, and the two LDS tile
// formats with their MFMA fragment readers.
#pragma once

#include "gm_device.h"

namespace gm {

typedef __attribute__((address_space(3))) void lds_void;
typedef short i16x4 __attribute__((ext_vector_type(4)));

// Sixteen zero bytes in global memory: the source of every DMA lane whose
// element lies outside the matrix or belongs to a pruned group.
extern __device__ __attribute__((aligned(16))) uint16_t g_zero_chunk[8];

// Pipeline depth (LDS stages) and K per stage.
constexpr int kStages = 4;
constexpr int kBK = 32;

// 16 bytes from global memory straight into LDS (global_load_lds_dwordx4):
// lane l of the wave writes lds_wave_base + 16 l.  lds_wave_base must be the
// same for the whole wave.  Issued through inline assembly so that the
// compiler does not add conservative waits for it; completion is tracked
// with wait_vmcnt() and made visible to the block with block_sync().  M0
// needs one wait state after it is written.  M0 is a reserved register the
// compiler cannot be told about; the kernels that use this helper have no
// other M0 reader (no GDS, message, move-relative or compiler-issued LDS DMA
// instructions), which the build's assembly check confirms.
__device__ __forceinline__ void dma16(const void* gsrc, const void* lds_wave_base) {
  const uint32_t l = uint32_t(reinterpret_cast<uintptr_t>((lds_void*)lds_wave_base));
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gsrc), "s"(__builtin_amdgcn_readfirstlane(l))
               : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most `pending` stages of `per_stage` DMA instructions are in flight.
template <int PER_STAGE>
__device__ __forceinline__ void wait_stages(int pending) {
  if (pending >= 2)
    wait_vmcnt<2 * PER_STAGE>();
  else if (pending == 1)
    wait_vmcnt<PER_STAGE>();
  else
    wait_vmcnt<0>();
}

// Workgroup barrier without the memory fence of __syncthreads (which would
// drain the in-flight DMA); the asm statements keep the compiler from moving
// LDS accesses across it.
__device__ __forceinline__ void block_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// ---------------------------------------------------------------- K-major tile
// R rows x 32 k, 64 bytes per row.  16-byte chunk c (k = 8c .. 8c+7) of row r
// sits at slot 4 r + (c ^ ((r >> 1) & 3)): eight consecutive rows read at one
// chunk cover all banks.

__device__ __forceinline__ int km_slot(int row, int chunk) { return row * 4 + (chunk ^ ((row >> 1) & 3)); }

// DMA slot s of the tile (s = 64 b + lane) -> (row, logical chunk).
__device__ __forceinline__ void km_dma_target(int s, int& row, int& chunk) {
  row = s >> 2;
  chunk = (s & 3) ^ ((row >> 1) & 3);
}

// MFMA fragment (8 consecutive k of one row) for lane l: row0 + (l & 15), k-chunk l >> 4.
__device__ __forceinline__ u32x4 km_frag(const u32x4* tile, int row0, int lane) {
  return tile[km_slot(row0 + (lane & 15), lane >> 4)];
}

// --------------------------------------------------------------- MN-major tile
// 32 k-rows x C columns (C = 64, 128 or 256), C*2 bytes per row.  16-byte chunk
// c of k-row r sits at slot r (C/8) + (c ^ 2 h(r)) with h(r) = (r & 3) | ((r >> 3) & 1) << 2
// (taken modulo C/16): the rows that one transposing read touches land on
// different 32-byte bank groups.

template <int C>
__device__ __forceinline__ int mn_h(int r) {
  return ((r & 3) | (((r >> 3) & 1) << 2)) & (C / 16 - 1);
}

template <int C>
__device__ __forceinline__ void mn_dma_target(int s, int& row, int& chunk) {
  constexpr int CPR = C / 8;  // chunks per row
  row = s / CPR;
  chunk = (s % CPR) ^ (2 * mn_h<C>(row));
}

// MFMA fragment for lane l from an MN-major tile: column col0 + (l & 15),
// k = 8 (l >> 4) .. 8 (l >> 4) + 7, assembled from two ds_read_b64_tr_b16.
// Within each 16-lane group the transposing read hands lane i element (i & 3)
// of the 8 bytes read by lane 4 q + (i >> 2), q = 0..3; lane j therefore reads
// the four columns col0 + 4 (j & 3) .. + 3 of k-row 8 G + (j >> 2).
template <int C>
__device__ __forceinline__ u32x4 mn_frag(const u32x4* tile, int col0, int lane) {
  const int i = lane & 15;
  const int r = 8 * (lane >> 4) + (i >> 2);
  const int slot32 = (col0 >> 4) ^ mn_h<C>(r);  // 32-byte unit within the row (h(r + 4) == h(r))
  const char* base = reinterpret_cast<const char*>(tile) + r * (C * 2) + slot32 * 32 + 8 * (i & 3);
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)base);
  const i16x4 hi =
      __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(base + 4 * C * 2));
  u32x4 f;
  __builtin_memcpy(&f, &lo, 8);
  __builtin_memcpy(reinterpret_cast<char*>(&f) + 8, &hi, 8);
  return f;
}

}  // namespace gm
