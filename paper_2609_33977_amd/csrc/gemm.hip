// bf16 MFMA GEMMs of the group-masked linear layer on gfx950.
//
//   fwd   Y[t, o]     = sum_v mask[u(o), v] sum_{i in v} X[t, i] W[o, i]        (Eq. 1)
//   dX    dX[t, i]    = sum_{o kept in column v(i)} mask[u(o), v] dY[t, o] W[o, i]
//   dgate dgate[u, v] = sum_{o in u, i in v} W[o, i] sum_t dY[t, o] X[t, i]
//
// Groups are g_out x g blocks (Sec. 2.1): u(o) = o / g_out is the mask row of
// output row o, v(i) = i / g its mask column; 1 x g groups have g_out = 1.
//
// Shared machinery (gm_gemm.h, gm_pipe.h): 256 x 256 output tiles (dX:
// min(max(g, 64), 256) x 256), eight waves of 128 x 64 (dX tiles of 64 rows:
// four waves of 32 x 128) accumulated in AGPRs and VGPRs with
// v_mfma_f32_16x16x32_bf16, and a four-stage pipeline of 32-deep K slices
// copied global -> LDS by buffer loads with the lds modifier (no registers in
// flight), with one block barrier per slice.  Each lane keeps a fixed 32-bit
// byte offset per copy; the K advance lives in the scalar buffer resource,
// and out-of-range offsets read zeros (padding, ragged tails, pruned groups).
// M is always the dimension that is contiguous in the output, so every lane
// stores 4 adjacent bf16 (8 bytes).
//
// Operand tiles:
//   fwd   W rows and X rows are K-contiguous: K-major tiles, ds_read_b128.
//         A pruned group is never read: its copy lanes get an out-of-range offset.
//         The K-loop visits only group columns that some row of the tile keeps.
//   dgate X and dY are stored [T, .]: K (= tokens) is the row index, so the
//         tiles are MN-major and fragments come from ds_read_b64_tr_b16.
//         Epilogue: the fp32 tile of X^T dY is multiplied by W and summed over
//         each group in registers and across lanes; dY^T X never reaches HBM.
//         The transposing reads of dY are 16-byte chunks of dY^T, which the
//         first row of tiles stores for the dX GEMM.
//   dX    K = the kept rows of one group column (its column list): whole rows
//         of W and of dY^T are gathered, MN-major tiles, transposing reads.
#include "gm_gemm.h"
#include "gm_launch.h"
#include "gm_lists.h"

namespace gm {

// Waves per block of the GEMMs: eight waves of 128 x 64 per 256 x 256 tile,
// two per SIMD, so one wave's copy issue and barrier wait hide behind the
// other's MFMAs.
constexpr int kFwdWaves = 8;
constexpr int kDgateWaves = 8;
constexpr int kDxWaves = 8;
// dX: 8 waves for tiles of 128 and 256 rows; the 64-row tile keeps 4 (its W
// slice is four copies, one per wave).
constexpr int dx_waves(int bm) { return bm >= 128 ? kDxWaves : 4; }

// LDS pipeline depth (K slices of kBK) per GEMM; the forward also keeps the
// tile's kept bits in LDS.
constexpr int kStagesDgate = 4;
constexpr int kStagesDx = 4;

// MFMA rows of a wave tile issued after each slice's barrier (the K-loop's RA):
// four for the forward and dgate (2.5-5 % faster than one), one for dX (level).
constexpr int kFwdRowsAfter = 4, kDgateRowsAfter = 4, kDxRowsAfter = 1;

// ============================================================================ fwd

// C[o, t] over K = d_in, tile 256 (o) x 256 (t); waves 2 (o) x 4 (t).
//
// The K-loop walks column units of U = max(g, 32) input columns (a 16-wide
// group shares its 32-deep slice with its neighbour) and visits only the
// units that some row of the tile keeps; inside a visited unit each 16-byte
// chunk of W whose group is pruned for its row is zero-filled instead of read.
//
// Split K (ksplit > 1, for launches with fewer tiles than half the CUs):
// block b works on tile b / ksplit and takes share b % ksplit of the tile's
// list of visited units (contiguous, in order), and stores its fp32 partial
// tile into part[share][t][o]; fwd_reduce_kernel then adds the shares in
// order and rounds once.
template <int G, int GO>
__global__ __launch_bounds__(64 * kFwdWaves) void fwd_kernel(const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
                                                  const float* __restrict__ mask, int T, int d_in, int d_out,
                                                  uint16_t* __restrict__ Y, int ksplit, float* __restrict__ part) {
  constexpr int NW = kFwdWaves, WN = NW / 2;  // waves per block; wave grid 2 (M) x WN (N)
  constexpr int BM = 256, BN = 256, MB = 8, NB = BN / WN / 16;
  constexpr int U = G < kBK ? kBK : G;        // input columns of one unit
  constexpr int UG = U / G;                   // groups per unit (2 for g = 16)
  constexpr int SUB = U / kBK;                // K slices per unit
  constexpr int RB = BM / GO;                 // mask rows met by one tile
  constexpr int MAXG = GO == 1 ? 512 : 1024;  // selectors per mask row (checked by the host)
  constexpr int MAXU = 512;                   // units per row (checked by the host)
  constexpr int PER_STAGE = 32 / NW;          // DMA instructions per wave per slice
  constexpr int CA = PER_STAGE / 2;           // of which copies of the W tile (the rest: X tile)
  constexpr int STAGES = 4;
  static_assert(GO == 1 || GO == G, "groups are 1 x g or square");
  __shared__ u32x4 As[STAGES][BM * 4];
  __shared__ u32x4 Bs[STAGES][BN * 4];
  __shared__ uint32_t s_bits[RB][MAXG / 32];  // kept bits of the tile's mask rows
  __shared__ uint32_t s_any[MAXU / 32];       // unit kept by some row of the tile
  __shared__ int s_cols[MAXU];
  __shared__ uint32_t s_live[GO >= 32 ? MAXU : 1];  // per listed unit: bit f = 16-row fragment f of the tile keeps it
  __shared__ int s_ncols, s_soft;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int G_in = d_in / G, NU = d_in / U;
  const int tiles_m = (d_out + BM - 1) / BM, tiles_n = (T + BN - 1) / BN;
  const int share = int(blockIdx.x) % ksplit;
  int tm, tn;
  tile_coords(int(blockIdx.x) / ksplit, int(gridDim.x) / ksplit, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;

  // Prologue: kept bits of every mask row of the tile, the units some row keeps, soft values.
  // The tile's RB mask rows are one contiguous run of RB * G_in selectors.
  // Pass 1 reads it coalesced, eight independent loads per thread at a time
  // (past the run or the layer's last mask row they read zeros), and stores
  // the kept flags as a flat bitmap, one ballot per 64 selectors, into the
  // first stage of the A tile, which the K-loop has not started to fill.
  if (tid < MAXU / 32) s_any[tid] = 0;
  if (tid == 0) {
    s_soft = 0;
    s_cols[0] = 0;  // read (unused) by the zero-fill copies when no unit is kept
  }
  uint32_t* flat = reinterpret_cast<uint32_t*>(&As[0][0]);
  {
    const int u0 = m0 / GO, rows = min(RB, d_out / GO - u0), n = RB * G_in;
    const __amdgpu_buffer_rsrc_t rm = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(mask + int64_t(u0) * G_in), short(0), rows * G_in * 4, 0x00020000);
    bool soft = false;
    for (int e0 = wave * 64; e0 < n; e0 += 8 * 64 * NW) {
      float m[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int e = e0 + i * 64 * NW + lane;
        m[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rm, e < n ? uint32_t(e) * 4u : kOOB, 0, 0));
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint64_t bal = __ballot(m[i] != 0.0f);
        soft |= m[i] != 0.0f && m[i] != 1.0f;
        const int e = e0 + i * 64 * NW;
        if (lane < 2 && e < n) flat[e / 32 + lane] = uint32_t(bal >> (32 * lane));
      }
    }
    __syncthreads();
    if (soft) s_soft = 1;
  }
  // Pass 2: word w of mask row r holds bits 32w .. 32w+31 of the row's G_in
  // (bits past the run are never extracted: a word stops at its row's end).
  {
    const int words = (G_in + 31) / 32;
    for (int e = tid; e < RB * words; e += 64 * NW) {
      const int r = e % RB, w = e / RB;
      const int p = r * G_in + 32 * w, nb = min(32, G_in - 32 * w);
      const uint64_t two = (uint64_t(flat[p / 32 + 1]) << 32) | flat[p / 32];
      const uint32_t b = uint32_t(two >> (p & 31)) & (nb == 32 ? ~0u : (1u << nb) - 1u);
      s_bits[r][w] = b;
      if constexpr (UG == 1) {
        if (b) atomicOr(&s_any[w], b);
      } else {
        // 16-wide groups: unit u holds groups 2u and 2u + 1; pack the pairs' ORs
        uint32_t u = (b | (b >> 1)) & 0x55555555u;
        u = (u | (u >> 1)) & 0x33333333u;
        u = (u | (u >> 2)) & 0x0f0f0f0fu;
        u = (u | (u >> 4)) & 0x00ff00ffu;
        u = (u | (u >> 8)) & 0x0000ffffu;
        if (u) atomicOr(&s_any[w >> 1], u << (16 * (w & 1)));
      }
    }
  }
  __syncthreads();
  if (wave == 0) {
    int cnt = 0;
    for (int ub = 0; ub < NU; ub += 64) {
      const int un = ub + lane;
      const bool f = un < NU && ((s_any[un >> 5] >> (un & 31)) & 1);
      const uint64_t bal = __ballot(f);
      if (f) {
        const int pos = cnt + __popcll(bal & ((uint64_t(1) << lane) - 1));
        s_cols[pos] = un;
        if constexpr (GO >= 32) {
          // square groups: all rows of a mask row share the unit's kept bits
          uint32_t live = 0;
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            uint32_t k = 0;
#pragma unroll
            for (int q = 0; q < UG; ++q) k |= s_bits[rb][(un * UG + q) >> 5] >> ((un * UG + q) & 31);
            if (k & 1u) live |= ((1u << (GO / 16)) - 1u) << (rb * (GO / 16));
          }
          s_live[pos] = live;
        }
      }
      cnt += __popcll(bal);
    }
    if (lane == 0) s_ncols = cnt;
  }
  __syncthreads();
  // this block's share of the visited units: list entries [c0, c1)
  const int c0 = share * s_ncols / ksplit, c1 = (share + 1) * s_ncols / ksplit;
  const int nst = (c1 - c0) * SUB;
  const int cb = c0 < s_ncols ? c0 : 0;  // an empty share reads (never consumes) entry 0
  const int* cols = s_cols + cb;

  // This lane's CA DMA rows (the same in both tiles): row = 16 (CA wave + j) + lane / 4,
  // their mask rows within the tile, the group of their chunk within a unit,
  // and their byte offsets within a K slice (out-of-range rows read zeros).
  int rowj[CA], brow[CA], gsub[CA];
  uint32_t offA[CA], offB[CA];
#pragma unroll
  for (int j = 0; j < CA; ++j) {
    int c;
    km_dma_target((wave * CA + j) * 64 + lane, rowj[j], c);
    brow[j] = rowj[j] / GO;
    gsub[j] = UG == 2 ? c >> 1 : 0;
    offA[j] = group_voffset(uint32_t((m0 + rowj[j]) * d_in + 8 * c) * 2u, j);
    offB[j] = group_voffset(uint32_t((n0 + rowj[j]) * d_in + 8 * c) * 2u, j);
  }
  const uint32_t bytesW = uint32_t(d_out) * uint32_t(d_in) * 2u;
  const uint32_t bytesX = uint32_t(T) * uint32_t(d_in) * 2u;

  // Per-slice copy state, set by prepare(): the buffer resources of the
  // slice's K range and the W offsets for its unit (chunks of pruned groups
  // get an out-of-range offset).  prepare() has no branches: the unit of the
  // next slice and the kept bits of this lane's chunks for it are read from
  // LDS one slice ahead, so their latency is hidden.
  const uint32_t ldsA = lds_addr(As), ldsB = lds_addr(Bs);
  auto col_of = [&](int st) { return st < nst ? st / SUB : 0; };  // slices past the end reuse unit 0
  auto group_of = [&](int un, int j) { return un * UG + gsub[j]; };
  int v_cur = __builtin_amdgcn_readfirstlane(cols[0]);
  int v_nxt = __builtin_amdgcn_readfirstlane(cols[col_of(1)]);
  // Square groups of 32 rows and more: fragment rows of this wave that keep
  // the unit of the slice consumed next (slice st - STAGES + 1 when
  // prepare(st) runs).  With 16 x 16 groups a fragment row skips a 32-deep
  // slice only when both of its groups are pruned, and the branches cost more
  // than the skipped MFMAs save, so every row runs.
  constexpr bool SKIP = GO >= 32;
  uint32_t live_nxt = ~0u;
  uint32_t bits_cur[CA];
#pragma unroll
  for (int j = 0; j < CA; ++j) bits_cur[j] = s_bits[brow[j]][group_of(v_cur, j) >> 5];
  uint32_t curA[CA];
  i32x4_t rA, rB;
  auto prepare = [&](int st) {
    const bool live = st < nst;
#pragma unroll
    for (int j = 0; j < CA; ++j) curA[j] = offA[j] | (((~bits_cur[j] >> (group_of(v_cur, j) & 31)) & 1u) << 31);
    const int k0 = live ? v_cur * U + (st % SUB) * kBK : 0;
    rA = make_rsrc_grouped(W + k0, live ? bytesW - 2u * uint32_t(k0) : 0u);
    rB = make_rsrc_grouped(X + k0, live ? bytesX - 2u * uint32_t(k0) : 0u);
#pragma unroll
    for (int j = 0; j < CA; ++j) bits_cur[j] = s_bits[brow[j]][group_of(v_nxt, j) >> 5];
    v_cur = v_nxt;
    v_nxt = __builtin_amdgcn_readfirstlane(cols[col_of(st + 2)]);
    if constexpr (SKIP)
      live_nxt = (__builtin_amdgcn_readfirstlane(s_live[cb + col_of(max(st - STAGES + 1, 0))]) >> (wm * 8)) & 0xffu;
  };
  auto live = [&](int) { return live_nxt; };
  // copies 0..CA-1 fill this wave's row blocks of the W tile, CA..2CA-1 of the X tile
  auto issue = [&](int st, int p) {
    const int j = p % CA;
    const uint32_t dst = (st % STAGES) * (BM * 64) + wave * CA * 1024;
    if (p < CA)
      dma16_group(j, rA, curA[j], ldsA + dst);
    else
      dma16_group(j, rB, offB[j], ldsB + dst);
  };
  // Soft selectors.  With every slice's copies, lane l of wave w also copies the
  // mask value of tile row 32 w + (l & 31) for the slice's unit (with 16-wide
  // groups: for the group of the slice's half l >> 5) into LDS; the wave's own
  // rows are exactly those rows, so after its copies land each lane scales its
  // W chunks by values its own wave brought in, with no extra wait.
  static_assert(CA * 16 == 32, "a wave copies the W chunks of 32 tile rows");
  __shared__ float s_msoft[STAGES][64 * NW];
  const i32x4_t rM = make_rsrc(mask, uint32_t(d_out / GO) * uint32_t(G_in) * 4u);
  const uint32_t ldsM = lds_addr(s_msoft) + uint32_t(wave) * 256u;
  auto prepare_soft = [&](int st) {
    const int r = 32 * wave + (lane & 31), h = lane >> 5;
    const bool ok = st < nst && m0 + r < d_out && (UG == 2 || h == 0);
    dma4_buf(rM, ok ? (uint32_t((m0 + r) / GO) * uint32_t(G_in) + uint32_t(v_cur * UG + h)) * 4u : kOOB,
             ldsM + uint32_t(st % STAGES) * (64u * NW * 4u));
    prepare(st);
  };
  auto rescale = [&](int st) {
    const float* ms = s_msoft[st % STAGES] + 64 * wave;
    u32x4* A = As[st % STAGES];
    float m[CA];
#pragma unroll
    for (int j = 0; j < CA; ++j) m[j] = ms[16 * j + (lane >> 2) + 32 * gsub[j]];
#pragma unroll
    for (int j = 0; j < CA; ++j) {
      u32x4* p = A + (wave * CA + j) * 64 + lane;
      if (m[j] != 0.0f && m[j] != 1.0f) *p = scale_bf16x8(*p, m[j]);
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  };

  // Hard masks (the common case) run a loop without the rescaling step.
  f32x4 acc[MB][NB];
  if (s_soft)
    gemm_mainloop<MB, NB, true, true, 0, 0, PER_STAGE, STAGES, kFwdRowsAfter, 1>(
        As, Bs, nst, wm * 128, wn * NB * 16, lane, acc, prepare_soft, issue, rescale, [](int, const u32x4(&)[NB]) {},
        live);
  else
    gemm_mainloop<MB, NB, true, true, 0, 0, PER_STAGE, STAGES, kFwdRowsAfter>(
        As, Bs, nst, wm * 128, wn * NB * 16, lane, acc, prepare, issue, [](int) {}, [](int, const u32x4(&)[NB]) {}, live);

  if (part) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int o = m0 + wm * 128 + mb * 16 + 4 * (lane >> 4);
        const int t = n0 + wn * NB * 16 + nb * 16 + (lane & 15);
        if (t < T && o < d_out) *reinterpret_cast<f32x4*>(part + (int64_t(share) * T + t) * d_out + o) = acc[mb][nb];
      }
    return;
  }
  store_tile_rows<BM, MB, NB, NW>(acc, reinterpret_cast<char*>(&As[0][0]), reinterpret_cast<char*>(&Bs[0][0]), wm, wn,
                                  tid, lane, Y, d_out, n0, T, m0, d_out);
}

// Y = bf16(sum over shares s = 0 .. ksplit-1 of part[s]), eight outputs per thread.
__global__ __launch_bounds__(256) void fwd_reduce_kernel(const float* __restrict__ part, int ksplit, int64_t n,
                                                         uint16_t* __restrict__ Y) {
  const int64_t e = (int64_t(blockIdx.x) * 256 + threadIdx.x) * 8;
  if (e >= n) return;
  f32x4 a = *reinterpret_cast<const f32x4*>(part + e), b = *reinterpret_cast<const f32x4*>(part + e + 4);
  for (int s = 1; s < ksplit; ++s) {
    a += *reinterpret_cast<const f32x4*>(part + int64_t(s) * n + e);
    b += *reinterpret_cast<const f32x4*>(part + int64_t(s) * n + e + 4);
  }
  uint4 w;
  w.x = pack_bf16x2(a[0], a[1]);
  w.y = pack_bf16x2(a[2], a[3]);
  w.z = pack_bf16x2(b[0], b[1]);
  w.w = pack_bf16x2(b[2], b[3]);
  *reinterpret_cast<uint4*>(Y + e) = w;
}

// ============================================================================ dgate

// C[i, o] = sum_t X[t, i] dY[t, o], tile 256 (i) x 256 (o); waves 2 (i) x 4 (o).
// The epilogue forms dgate[o, v] = sum_{i in v} W[o, i] C[i, o].  For g = 512 a
// group spans two tiles, each adding its half onto a zeroed dgate (two
// addends onto zero: the same sum whichever lands first).
//
// Blocks past the tiles (when the dX GEMM follows) build the mask's column
// lists, one col_lists_unit each: they start as the first tiles finish, on
// CUs that would otherwise idle through the last tiles' tail (or a partial
// last round of tiles), instead of in a launch of their own before dgate.
struct ListArgs {
  const float* mask;
  int nunits, nchunks, nsub;
  int *colcount, *colsoft, *rows, *subbits;
  float* scales;
};

template <int G, int GO>
__global__ __launch_bounds__(64 * kDgateWaves) void dgate_kernel(const uint16_t* __restrict__ dY, const uint16_t* __restrict__ X,
                                                    const uint16_t* __restrict__ W, int T, int d_in, int d_out,
                                                    float* __restrict__ dgate, uint16_t* __restrict__ dYt, int ldt,
                                                    ListArgs la) {
  constexpr int NW = kDgateWaves, WN = NW / 2;  // waves per block; wave grid 2 (i) x WN (o)
  constexpr int BM = 256, BN = 256, MB = 8, NB = BN / WN / 16;
  constexpr int PER_STAGE = 32 / NW;
  constexpr int CA = PER_STAGE / 2;  // copies of the X tile per wave (the rest: dY tile)
  constexpr int STAGES = kStagesDgate;
  __shared__ u32x4 As[STAGES][kBK * BM / 8];
  __shared__ u32x4 Bs[STAGES][kBK * BN / 8];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int G_in = d_in / G;
  const int tiles_m = (d_in + BM - 1) / BM, tiles_n = (d_out + BN - 1) / BN, tiles = tiles_m * tiles_n;
  if (int(blockIdx.x) >= tiles) {
    col_lists_unit<64 * NW>(int(blockIdx.x) - tiles, la.nchunks, la.mask, d_out, G_in, GO, la.nsub, la.colcount,
                            la.colsoft, la.rows, la.scales, la.subbits);
    return;
  }
  int tm, tn;
  tile_coords(int(blockIdx.x), tiles, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int nst = (T + kBK - 1) / kBK;

  // Byte offsets of this lane's DMA chunks within a K slice (columns past the
  // matrix read zeros; rows past T fall outside the slice's range).
  uint32_t offA[CA], offB[CA];
#pragma unroll
  for (int j = 0; j < CA; ++j) {
    int row, c;
    mn_dma_target<256>((wave * CA + j) * 64 + lane, row, c);
    offA[j] = group_voffset(m0 + 8 * c < d_in ? uint32_t(row * d_in + m0 + 8 * c) * 2u : kOOB, j);
    offB[j] = group_voffset(n0 + 8 * c < d_out ? uint32_t(row * d_out + n0 + 8 * c) * 2u : kOOB, j);
  }
  const uint32_t bytesX = uint32_t(T) * uint32_t(d_in) * 2u;
  const uint32_t bytesY = uint32_t(T) * uint32_t(d_out) * 2u;
  i32x4_t rA, rB;  // buffer resources of the slice being copied (zero length past the end)
  auto prepare = [&](int st) {
    const bool live = st < nst;
    const int k0 = live ? st * kBK : 0;
    rA = make_rsrc_grouped(X + int64_t(k0) * d_in, live ? bytesX - uint32_t(k0) * uint32_t(d_in) * 2u : 0u);
    rB = make_rsrc_grouped(dY + int64_t(k0) * d_out, live ? bytesY - uint32_t(k0) * uint32_t(d_out) * 2u : 0u);
  };
  const uint32_t ldsA = lds_addr(As), ldsB = lds_addr(Bs);
  auto issue = [&](int st, int p) {
    const int j = p % CA;
    const uint32_t dst = (st % STAGES) * (kBK * BM * 2) + wave * CA * 1024;
    if (p < CA)
      dma16_group(j, rA, offA[j], ldsA + dst);
    else
      dma16_group(j, rB, offB[j], ldsB + dst);
  };

  // dY^T side output (for the dX GEMM): lane (G, i) of a B fragment holds
  // dY[k0 + 8 G .. k0 + 8 G + 7, o] for o = n0 + wn*NB*16 + nb*16 + i, which is a
  // 16-byte chunk of row o of dY^T.  The tiles sharing this dY panel split
  // the slices between them (slice kt goes to tile row kt * tiles_m / nst), and
  // within a tile the two wave rows, which hold the same B fragments, alternate.
  auto bhook = [&](int kt, const u32x4(&bf)[NB]) {
    if (dYt == nullptr || (kt * tiles_m) / nst != tm || (kt & 1) != wm) return;
    const int t = kt * kBK + 8 * (lane >> 4);
    if (t >= ldt) return;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int o = n0 + wn * NB * 16 + nb * 16 + (lane & 15);
      if (o < d_out) st16(dYt + int64_t(o) * ldt + t, bf[nb]);
    }
  };

  f32x4 acc[MB][NB];
  gemm_mainloop<MB, NB, false, false, BM, BN, PER_STAGE, STAGES, kDgateRowsAfter>(
      As, Bs, nst, wm * 128, wn * NB * 16, lane, acc, prepare, issue, [](int) {}, bhook);

  // Epilogue.  Lane (l >> 4, l & 15) holds, for every (mb, nb), rows
  // i = i0 .. i0 + 3 of column o: W[o, i0 .. i0 + 3] is one 8-byte load.
  const int ibase = m0 + wm * 128 + 4 * (lane >> 4);
  if constexpr (GO > 1) {
    // Square groups (GO = G = 16 .. 128): a 16 x 16 fragment lies inside one
    // group, so each lane sums its products per group of the wave's 128 (i) x
    // 64 (o) sub-tile, and one reduction over the 64 lanes finishes the wave's
    // share of each group.  Groups of 128 rows span two waves (wn pairs),
    // which add their halves in a fixed order through LDS.
    constexpr int IB = 128 / G;                  // groups along i in a wave
    constexpr int OS = GO < 64 ? 64 / GO : 1;    // groups (or group halves) along o in a wave
    float part[IB][OS];
#pragma unroll
    for (int a = 0; a < IB; ++a)
#pragma unroll
      for (int b = 0; b < OS; ++b) part[a][b] = 0.0f;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int o = n0 + wn * NB * 16 + nb * 16 + (lane & 15);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const int i0 = ibase + mb * 16;
        if (o < d_out && i0 < d_in) {
          const uint2 w = *reinterpret_cast<const uint2*>(W + int64_t(o) * d_in + i0);
          part[mb * 16 / G][nb * 16 / (GO < 64 ? GO : 64)] +=
              acc[mb][nb][0] * bf16_lo(w.x) + acc[mb][nb][1] * bf16_hi(w.x) + acc[mb][nb][2] * bf16_lo(w.y) +
              acc[mb][nb][3] * bf16_hi(w.y);
        }
      }
    }
#pragma unroll
    for (int a = 0; a < IB; ++a)
#pragma unroll
      for (int b = 0; b < OS; ++b) {
        float x = part[a][b];
#pragma unroll
        for (int d = 32; d >= 1; d >>= 1) x += __shfl_xor(x, d);
        part[a][b] = x;
      }
    const int G_out = d_out / GO;
    if constexpr (GO < 128) {
      if (lane == 0) {
#pragma unroll
        for (int a = 0; a < IB; ++a)
#pragma unroll
          for (int b = 0; b < OS; ++b) {
            const int v = (m0 + wm * 128) / G + a;
            const int u = (n0 + wn * 64) / GO + b;
            if (u < G_out && v < G_in) dgate[int64_t(u) * G_in + v] = part[a][b];
          }
      }
    } else {
      float* s_half = reinterpret_cast<float*>(&As[0][0]);
      __syncthreads();  // every wave has left its K-loop (copies drained)
      if (lane == 0) s_half[wave] = part[0][0];
      __syncthreads();
      if (tid < 4) {  // group (a, b) of the tile: waves (a, 2b) and (a, 2b + 1)
        const int a = tid >> 1, b = tid & 1;
        const int u = n0 / GO + b, v = m0 / G + a;
        if (u < G_out && v < G_in) dgate[int64_t(u) * G_in + v] = s_half[a * WN + 2 * b] + s_half[a * WN + 2 * b + 1];
      }
    }
  } else {
    float part[NB][2];  // per o column: group sums over this wave's first / second 64 rows of i
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int o = n0 + wn * NB * 16 + nb * 16 + (lane & 15);
      float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const int i0 = ibase + mb * 16;
        if (o < d_out && i0 < d_in) {
          const uint2 w = *reinterpret_cast<const uint2*>(W + int64_t(o) * d_in + i0);
          const float s = acc[mb][nb][0] * bf16_lo(w.x) + acc[mb][nb][1] * bf16_hi(w.x) +
                          acc[mb][nb][2] * bf16_lo(w.y) + acc[mb][nb][3] * bf16_hi(w.y);
          if (mb < MB / 2) s0 += s; else s1 += s;
        }
      }
      // sum over the four lane groups (they hold the other i of the same o)
      s0 += __shfl_xor(s0, 16);
      s0 += __shfl_xor(s0, 32);
      s1 += __shfl_xor(s1, 16);
      s1 += __shfl_xor(s1, 32);
      part[nb][0] = s0;
      part[nb][1] = s1;
    }
    if constexpr (G == 64) {
      if (lane < 16) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int o = n0 + wn * NB * 16 + nb * 16 + lane;
          const int v = (m0 + wm * 128) / 64;
          if (o < d_out && v < G_in) dgate[int64_t(o) * G_in + v] = part[nb][0];
          if (o < d_out && v + 1 < G_in) dgate[int64_t(o) * G_in + v + 1] = part[nb][1];
        }
      }
    } else if constexpr (G == 128) {
      if (lane < 16) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int o = n0 + wn * NB * 16 + nb * 16 + lane;
          const int v = (m0 + wm * 128) / 128;
          if (o < d_out && v < G_in) dgate[int64_t(o) * G_in + v] = part[nb][0] + part[nb][1];
        }
      }
    } else {
      // The two wave rows combine through LDS, reusing the first stage buffer
      // once every wave has finished its K-loop (their copies have drained).
      float(*s_part)[BN] = reinterpret_cast<float(*)[BN]>(&As[0][0]);
      __syncthreads();
      if (lane < 16) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) s_part[wm][wn * NB * 16 + nb * 16 + lane] = part[nb][0] + part[nb][1];
      }
      __syncthreads();
      const int o = n0 + tid;
      if (tid < BN && o < d_out) {
        const float h = s_part[0][tid] + s_part[1][tid];
        if constexpr (G == 256)
          dgate[int64_t(o) * G_in + m0 / 256] = h;
        else
          atomicAdd(dgate + int64_t(o) * G_in + m0 / 512, h);
      }
    }
  }
}

// Fill n floats with zero (before the order-independent two-tile accumulation).
__global__ __launch_bounds__(256) void zero_f32_kernel(float* __restrict__ p, int64_t n) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0.0f;
}

// ============================================================================ dX

// C[i, t] = sum_k W[o_k, i] dYt[o_k, t] over the listed rows o_k of list
// column v (lc = max(g, 64) input columns), tile BM (i, BM = min(lc, 256)) x
// 256 (t); waves 2 (i) x WN (t).  The column list is read with scalar loads
// (KR entries per wave per slice), one slice ahead of its DMA.  With NSUB > 1
// (groups of 16 or 32 columns) a list column holds NSUB groups and lists
// every row that keeps one of them; each entry carries its kept bits, and the
// 16-byte chunks of W in a pruned group are zero-filled instead of read.
template <int BM, int NSUB>
__global__ __launch_bounds__(64 * dx_waves(BM)) void dx_kernel(const uint16_t* __restrict__ dYt, int ldt,
                                                 const uint16_t* __restrict__ W, const int* __restrict__ colcount,
                                                 const int* __restrict__ rows, const float* __restrict__ scales,
                                                 const int* __restrict__ subbits, const int* __restrict__ colsoft,
                                                 int T, int d_in, int d_out, int lc, uint16_t* __restrict__ dX) {
  constexpr int NW = dx_waves(BM), WN = NW / 2;  // waves per block; wave grid 2 (i) x WN (t)
  constexpr int BN = 256, MB = BM / 32, NB = BN / WN / 16;
  constexpr int KR = kBK / NW;               // k-rows of a slice gathered by one wave
  constexpr int NA = BM / 16 / NW;           // A DMA instructions per wave per slice
  constexpr int NBC = BN / 16 / NW;          // B DMA instructions per wave per slice
  constexpr int PER_STAGE = NA + NBC;
  constexpr int STAGES = kStagesDx;
  __shared__ u32x4 As[STAGES][kBK * BM / 8];
  __shared__ u32x4 Bs[STAGES][kBK * BN / 8];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int tiles_m = d_in / BM, tiles_n = (T + BN - 1) / BN;
  int tm, tn;
  tile_coords(gridDim.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int v = m0 / lc;
  const int kv = colcount[v];
  const bool soft = colsoft[v] != 0;
  const int* __restrict__ rl = rows + int64_t(v) * d_out;
  const int* __restrict__ bl = subbits + int64_t(v) * d_out;
  const float* __restrict__ sl = scales + int64_t(v) * d_out * NSUB;
  const int nst = (kv + kBK - 1) / kBK;
  constexpr int CPS = BM / 8 / NSUB;  // 16-byte chunks per group along i (NSUB > 1)

  // Slice st uses k-rows st*32 + r; this wave gathers rows r = KR wave .. KR wave + KR - 1,
  // whose list entries are read with scalar loads one slice ahead.
  int idx[KR], kbits[NSUB > 1 ? KR : 1];
  auto load_idx = [&](int st) {  // st <= nst: at most 31 + 32 entries past the column's end
    const int base = st * kBK + wave * KR;
#pragma unroll
    for (int q = 0; q < KR; ++q) {
      idx[q] = rl[base + q];  // uniform: scalar loads
      if constexpr (NSUB > 1) kbits[q] = bl[base + q];
    }
  };
  // Copy j of a wave in a tile with C columns (CPR = C / 8 chunks per k-row)
  // covers k-rows KR wave + j * RPI + lane / CPR, RPI = 64 / CPR: the lane's
  // row is one of RPI consecutive list entries of the wave.
  // The entries are wave-uniform.  For chains of more than two, passing them
  // through readfirstlane keeps the compiler from turning the selects into a
  // per-lane indexed load from a stack copy of the array (for two it emits
  // one select, and the extra moves would only cost VALU issue slots).
  auto pick_in = [&](const int* a, int j, auto rpi_c, int u) {
    constexpr int rpi = decltype(rpi_c)::value;
    auto entry = [&](int q) { return rpi > 2 ? __builtin_amdgcn_readfirstlane(a[j * rpi + q]) : a[j * rpi + q]; };
    int o = entry(0);
#pragma unroll
    for (int q = 1; q < rpi; ++q) o = u == q ? entry(q) : o;
    return o;
  };
  auto pick = [&](int j, auto rpi_c, int u) { return pick_in(idx, j, rpi_c, u); };
  constexpr std::integral_constant<int, 512 / BM> RPI_A{};
  constexpr std::integral_constant<int, 512 / BN> RPI_B{};
  const i32x4_t rA = make_rsrc_grouped(W + m0, (uint32_t(d_out) * uint32_t(d_in) - uint32_t(m0)) * 2u);
  const i32x4_t rB = make_rsrc_grouped(dYt + n0, (uint32_t(d_out) * uint32_t(ldt) - uint32_t(n0)) * 2u);
  uint32_t offA[NA], offB[NBC];  // this slice's per-lane offsets (rows past the list read zeros)
  auto prepare = [&](int st) {
    const int k0 = st * kBK;
#pragma unroll
    for (int j = 0; j < NA; ++j) {
      int row, c;
      mn_dma_target<BM>((wave * NA + j) * 64 + lane, row, c);
      const int o = pick(j, RPI_A, lane / (BM / 8));
      bool dead = k0 + row >= kv;
      if constexpr (NSUB > 1) dead |= ((pick_in(kbits, j, RPI_A, lane / (BM / 8)) >> (c / CPS)) & 1) == 0;
      offA[j] = group_voffset(uint32_t(o * d_in + 8 * c) * 2u | uint32_t(dead) << 31, j);
    }
#pragma unroll
    for (int j = 0; j < NBC; ++j) {
      int row, c;
      mn_dma_target<BN>((wave * NBC + j) * 64 + lane, row, c);
      const int o = pick(j, RPI_B, lane / (BN / 8));
      offB[j] = group_voffset(uint32_t(o * ldt + 8 * c) * 2u | uint32_t(k0 + row >= kv || n0 + 8 * c >= ldt) << 31, j);
    }
    load_idx(min(st + 1, nst));
  };
  const uint32_t ldsA = lds_addr(As), ldsB = lds_addr(Bs);
  auto issue = [&](int st, int p) {  // copies 0 .. NA-1: W tile, NA .. NA+NBC-1: dY^T tile
    if (p < NA)
      dma16_group(p, rA, offA[p], ldsA + (st % STAGES) * (kBK * BM * 2) + wave * NA * 1024);
    else
      dma16_group(p - NA, rB, offB[p - NA], ldsB + (st % STAGES) * (kBK * BN * 2) + wave * NBC * 1024);
  };
  // Soft selectors: scale this lane's landed W chunks by the row's mask value.
  auto rescale = [&](int st) {
    const int k0 = st * kBK;
    u32x4* A = As[st % STAGES];
#pragma unroll
    for (int j = 0; j < NA; ++j) {
      const int b = wave * NA + j;
      int row, c;
      mn_dma_target<BM>(b * 64 + lane, row, c);
      if (k0 + row < kv) {
        const float s = NSUB > 1 ? sl[(k0 + row) * NSUB + c / CPS] : sl[k0 + row];
        u32x4* p = A + b * 64 + lane;
        if (s != 1.0f) *p = scale_bf16x8(*p, s);
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  };

  // Columns whose kept selectors are all exactly 1 run a loop without the rescaling step.
  f32x4 acc[MB][NB];
  load_idx(0);
  if (soft)
    gemm_mainloop<MB, NB, false, false, BM, BN, PER_STAGE, STAGES, kDxRowsAfter>(
        As, Bs, nst, wm * (BM / 2), wn * NB * 16, lane, acc, prepare, issue, rescale, [](int, const u32x4(&)[NB]) {});
  else
    gemm_mainloop<MB, NB, false, false, BM, BN, PER_STAGE, STAGES, kDxRowsAfter>(
        As, Bs, nst, wm * (BM / 2), wn * NB * 16, lane, acc, prepare, issue, [](int) {}, [](int, const u32x4(&)[NB]) {});

  char* const hi = reinterpret_cast<char*>(&Bs[0][0]);
  store_tile_rows<BM, MB, NB, NW>(acc, BM == 256 ? reinterpret_cast<char*>(&As[0][0]) : hi, hi, wm, wn, tid, lane, dX,
                                  d_in, n0, T, m0, d_in);
}

// ============================================================================ dY^T

// dY [T, d_out] -> dYt [d_out, ldt] (t in [T, ldt) zero).  One 8 x 8 block per thread.
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

// The group shapes built: 1 x {64, 128, 256, 512} and square {16, 32, 64, 128}.
#define GM_CASE_G(KERNEL, G, GO, GRID, THREADS, ...) \
  case (G << 8) | GO: hipLaunchKernelGGL((KERNEL<G, GO>), dim3(GRID), dim3(THREADS), 0, s, __VA_ARGS__); break;
#define GM_LAUNCH_G(KERNEL, GRID, THREADS, ...)                  \
  switch ((g << 8) | go) {                                       \
    GM_CASE_G(KERNEL, 64, 1, GRID, THREADS, __VA_ARGS__)         \
    GM_CASE_G(KERNEL, 128, 1, GRID, THREADS, __VA_ARGS__)        \
    GM_CASE_G(KERNEL, 256, 1, GRID, THREADS, __VA_ARGS__)        \
    GM_CASE_G(KERNEL, 512, 1, GRID, THREADS, __VA_ARGS__)        \
    GM_CASE_G(KERNEL, 16, 16, GRID, THREADS, __VA_ARGS__)        \
    GM_CASE_G(KERNEL, 32, 32, GRID, THREADS, __VA_ARGS__)        \
    GM_CASE_G(KERNEL, 64, 64, GRID, THREADS, __VA_ARGS__)        \
    GM_CASE_G(KERNEL, 128, 128, GRID, THREADS, __VA_ARGS__)      \
    default: return hipErrorInvalidValue;                        \
  }

hipError_t launch_fwd(const uint16_t* X, const uint16_t* W, const float* mask, int T, int d_in, int d_out, int g,
                      int go, uint16_t* Y, int ksplit, float* part, hipStream_t s) {
  if (ksplit < 1 || (ksplit > 1 && part == nullptr)) return hipErrorInvalidValue;
  const int tiles = ((T + 255) / 256) * ((d_out + 255) / 256);
  float* p = ksplit > 1 ? part : nullptr;
  GM_LAUNCH_G(fwd_kernel, tiles * ksplit, 64 * kFwdWaves, X, W, mask, T, d_in, d_out, Y, ksplit, p)
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || ksplit == 1) return e;
  const int64_t n = int64_t(T) * d_out;  // a multiple of 8 (d_out is)
  hipLaunchKernelGGL(fwd_reduce_kernel, dim3(unsigned((n / 8 + 255) / 256)), dim3(256), 0, s, part, ksplit, n, Y);
  return hipGetLastError();
}

hipError_t launch_dgate(const uint16_t* dY, const uint16_t* X, const uint16_t* W, int T, int d_in, int d_out, int g,
                        int go, float* dgate, uint16_t* dYt, int ldt, const float* mask, int nsub, int* colcount,
                        int* colsoft, int* rows, float* scales, int* subbits, hipStream_t s) {
  const int tiles = ((d_out + 255) / 256) * ((d_in + 255) / 256);
  ListArgs la{mask, 0, (d_out + kListChunk - 1) / kListChunk, nsub, colcount, colsoft, rows, subbits, scales};
  if (colcount) la.nunits = (d_in / g / nsub) * la.nchunks;
  if (g == 512) {
    const int64_t n = int64_t(d_out) * (d_in / g);
    const unsigned blocks = unsigned(n / 256 + 1 < 4096 ? n / 256 + 1 : 4096);
    hipLaunchKernelGGL(zero_f32_kernel, dim3(blocks), dim3(256), 0, s, dgate, n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  GM_LAUNCH_G(dgate_kernel, tiles + la.nunits, 64 * kDgateWaves, dY, X, W, T, d_in, d_out, dgate, dYt, ldt, la)
  return hipGetLastError();
}

hipError_t launch_transpose(const uint16_t* dY, int T, int d_out, uint16_t* dYt, int ldt, hipStream_t s) {
  const int64_t nblk = int64_t(ldt / 8) * (d_out / 8);
  hipLaunchKernelGGL(transpose_kernel, dim3(unsigned((nblk + 255) / 256)), dim3(256), 0, s, dY, T, d_out, dYt, ldt);
  return hipGetLastError();
}

hipError_t launch_dx(const uint16_t* dYt, int ldt, const uint16_t* W, const int* colcount, const int* rows,
                     const float* scales, const int* subbits, const int* colsoft, int T, int d_in, int d_out, int g,
                     uint16_t* dX, hipStream_t s) {
  const int lc = g < 64 ? 64 : g;  // list-column width
  int bm = lc < 256 ? lc : 256;
  // A launch of fewer than 64 tiles (the 128-token, 1024 x 1024 linear has 4)
  // takes tiles of 64 columns, four times as many blocks over the same lists.
  if (g >= 64 && bm > 64 && (d_in / bm) * ((T + 255) / 256) < 64) bm = 64;
  const int tiles = (d_in / bm) * ((T + 255) / 256);
#define GM_DX(BM, NSUB)                                                                                        \
  hipLaunchKernelGGL((dx_kernel<BM, NSUB>), dim3(tiles), dim3(64 * dx_waves(BM)), 0, s, dYt, ldt, W, colcount, \
                     rows, scales, subbits, colsoft, T, d_in, d_out, lc, dX)
  switch (g) {
    case 16: GM_DX(64, 4); break;
    case 32: GM_DX(64, 2); break;
    case 64: GM_DX(64, 1); break;
    case 128:
      if (bm == 64) GM_DX(64, 1); else GM_DX(128, 1);
      break;
    case 256:
    case 512:
      if (bm == 64) GM_DX(64, 1); else GM_DX(256, 1);
      break;
    default: return hipErrorInvalidValue;
  }
#undef GM_DX
  return hipGetLastError();
}

}  // namespace gm
