// Building blocks of the pipelined LDS GEMMs on gfx950: asynchronous
// global -> LDS copies, explicit memory-counter waits, and the two LDS tile
// formats with their MFMA fragment readers.
#pragma once

#include "gm_device.h"

namespace gm {

typedef __attribute__((address_space(3))) void lds_void;
typedef short i16x4 __attribute__((ext_vector_type(4)));

// K per LDS pipeline stage.
constexpr int kBK = 32;

// Copies go from global memory straight into LDS with buffer loads (below),
// issued through inline assembly so that the compiler does not add
// conservative waits for them; completion is tracked with wait_vmcnt() and
// made visible to the block with block_sync().  The LDS destination is taken
// from M0, which needs one wait state after it is written.  M0 is a reserved
// register the compiler cannot be told about; the kernels that use these
// helpers have no other M0 reader (no GDS, message, move-relative or
// compiler-issued LDS DMA instructions).

// Buffer resource over a byte range [base, base + bytes): loads at offsets
// outside it return zeros, which is how the kernels read padding, ragged
// tails and pruned groups without branches.
typedef int32_t i32x4_t __attribute__((ext_vector_type(4)));
constexpr uint32_t kOOB = 0x80000000u;  // an offset past every range (ranges stay below 2 GiB)

__device__ __forceinline__ i32x4_t make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  i32x4_t r;
  r[0] = int32_t(uint32_t(b));
  r[1] = int32_t(uint32_t(b >> 32) & 0xffffu);  // stride 0: raw byte buffer
  r[2] = int32_t(bytes);
  r[3] = 0x00020000;
  r[0] = __builtin_amdgcn_readfirstlane(r[0]);
  r[1] = __builtin_amdgcn_readfirstlane(r[1]);
  r[2] = __builtin_amdgcn_readfirstlane(r[2]);
  return r;
}

// 32-bit LDS byte address of a __shared__ object (computed once per kernel:
// the generic -> LDS conversion checks for null).
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(uint32_t(reinterpret_cast<uintptr_t>((lds_void*)p)));
}

// buffer_load_dwordx4 (or _dword) ... offen lds copies 16 (or 4) bytes per
// lane from rsrc + voffset into LDS at M0 + 16 lane (or 4 lane), zeros when
// voffset is out of the resource's range (ranges stay below 2 GiB, so setting
// bit 31 of an offset marks it out of range).  M0 holds an LDS byte address,
// uniform across the wave.

// Grouped copies: up to four copies J = 0..3 of a wave share one M0 value.
// The instruction offset of buffer_load ... lds adds to both the memory
// offset and the LDS address, so copy J uses offset 1024 J and lands at
// m0 + 1024 J + 16 lane.  To keep every lane's memory offset non-negative,
// the buffer resource starts kDmaBias bytes early (make_rsrc_grouped) and
// copy J's lane offset is biased by kDmaBias - 1024 J (group_voffset); the
// range check is unchanged, and an offset with bit 31 set stays out of range.
constexpr uint32_t kDmaBias = 3072;

__device__ __forceinline__ i32x4_t make_rsrc_grouped(const void* base, uint32_t bytes) {
  return make_rsrc(static_cast<const char*>(base) - kDmaBias, bytes + kDmaBias);
}

__device__ __forceinline__ uint32_t group_voffset(uint32_t off, int j) { return off + kDmaBias - 1024u * uint32_t(j); }

// Copy J of a group; J == 0 sets M0 to the group's LDS base (uniform).
template <int J>
__device__ __forceinline__ void dma16_group(i32x4_t rsrc, uint32_t voffset, uint32_t lds_group_base) {
  static_assert(J >= 0 && J < 4, "four copies per M0 value");
  if constexpr (J == 0)
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
                 :
                 : "v"(voffset), "s"(rsrc), "s"(lds_group_base)
                 : "memory");
  else
    asm volatile("buffer_load_dwordx4 %0, %1, 0 offen offset:%2 lds" : : "v"(voffset), "s"(rsrc), "n"(J * 1024) : "memory");
}

__device__ __forceinline__ void dma16_group(int j, i32x4_t rsrc, uint32_t voffset, uint32_t lds_group_base) {
  switch (j) {
    case 0: dma16_group<0>(rsrc, voffset, lds_group_base); break;
    case 1: dma16_group<1>(rsrc, voffset, lds_group_base); break;
    case 2: dma16_group<2>(rsrc, voffset, lds_group_base); break;
    default: dma16_group<3>(rsrc, voffset, lds_group_base); break;
  }
}

// One 4-byte copy per lane into LDS at lds_wave_base + 4 lane.  It sets M0, so
// it must not sit between the copies of a group (dma16_group<J > 0> reuse M0).
__device__ __forceinline__ void dma4_buf(i32x4_t rsrc, uint32_t voffset, uint32_t lds_wave_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dword %0, %1, 0 offen lds"
               :
               : "v"(voffset), "s"(rsrc), "s"(lds_wave_base)
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
// sits at slot 4 r + (c ^ ((r >> 1) & 3)).  A 16-byte-per-lane LDS read is
// served eight lanes (128 bytes) per cycle: the eight consecutive rows that
// eight lanes of one fragment read touch occupy two 64-byte row pairs, and the
// XOR with bits 1-2 of the row moves rows of equal parity to four different
// 16-byte columns, so the eight lanes cover the 128 bytes once.  The XOR term
// depends only on the row within its 16-row fragment, so fragment addresses
// are a per-lane base plus compile-time offsets.

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
