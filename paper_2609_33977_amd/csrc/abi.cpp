// C-ABI layer of libgroupmask: argument validation, workspace planning and
// dispatch to the gfx950 kernels.  Nothing here allocates device memory, and
// every entry point checks all of its arguments before the first launch.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>

#include "../../include/groupmask.h"
#include "gm_launch.h"

#define GM_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

constexpr int64_t kMaxDim = int64_t(1) << 30;  // kernels index rows and columns with 32-bit ints
constexpr int kMaxUnits = 512;                 // forward GEMM: column units (max(g, 32) wide) per row
constexpr int kDecodeTokens = 16;              // forward dispatch: T <= 16 takes the GEMV path
constexpr int64_t kMaxElems = (int64_t(1) << 30) - (int64_t(1) << 22);  // bf16 elements per matrix (< 2 GiB)

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned8(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Debug modes, read once from the environment variable GM_DEBUG:
//   unset   no reporting;
//   "sync"  every launch is followed by a device-wide synchronisation and an
//           error check, so a fault is reported by the entry point that caused
//           it (GM_ERR_DEVICE) instead of by a later call (not for use under
//           graph capture);
//   other   the HIP error behind a GM_ERR_DEVICE status is printed to stderr
//           (also in "sync" mode).
int debug_mode() {
  static const int mode = [] {
    const char* v = std::getenv("GM_DEBUG");
    if (v == nullptr) return 0;
    return std::strcmp(v, "sync") == 0 ? 2 : 1;
  }();
  return mode;
}

gm_status device_error(const char* what, hipError_t e) {
  if (debug_mode()) std::fprintf(stderr, "libgroupmask: %s: HIP error %d (%s)\n", what, int(e), hipGetErrorName(e));
  return GM_ERR_DEVICE;
}

// gfx950 check, cached per device.
gm_status check_device() {
  static std::mutex mu;
  static signed char ok[256];  // 0 unknown, 1 yes, -1 no
  int dev = 0;
  if (hipError_t e = hipGetDevice(&dev)) return device_error("hipGetDevice", e);
  if (dev < 0 || dev >= 256) return device_error("device index", hipErrorInvalidDevice);
  std::lock_guard<std::mutex> lock(mu);
  if (ok[dev] == 0) {
    hipDeviceProp_t prop;
    if (hipError_t e = hipGetDeviceProperties(&prop, dev)) return device_error("hipGetDeviceProperties", e);
    ok[dev] = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : -1;
  }
  return ok[dev] == 1 ? GM_OK : device_error("not a gfx950 device", hipErrorInvalidDevice);
}

gm_status from_hip(hipError_t e) {
  if (e != hipSuccess) return device_error("kernel launch", e);
  if (debug_mode() == 2) {
    if (hipError_t s = hipDeviceSynchronize()) return device_error("kernel execution (GM_DEBUG=sync)", s);
    if (hipError_t s = hipGetLastError()) return device_error("after synchronisation (GM_DEBUG=sync)", s);
  }
  return GM_OK;
}

gm_status check_tau(float tau) { return (std::isfinite(tau) && tau > 0.0f) ? GM_OK : GM_ERR_VALUE; }

// Group shapes built: 1 x {64, 128, 256, 512} and square {16, 32, 64, 128}.
bool group_shape_ok(int32_t g, int32_t g_out) {
  if (g_out == 1) return g == 64 || g == 128 || g == 256 || g == 512;
  return g_out == g && (g == 16 || g == 32 || g == 64 || g == 128);
}

// Width of a column unit of the forward GEMM and of a list column of dX.
int64_t unit_width(int32_t g) { return g < 32 ? 32 : g; }
int64_t list_width(int32_t g) { return g < 64 ? 64 : g; }

gm_status check_linear_shape(int64_t T, int64_t d_in, int64_t d_out, int32_t g, int32_t g_out) {
  if (T < 1 || d_in < 1 || d_out < 1) return GM_ERR_SHAPE;
  if (T > kMaxDim || d_in > kMaxDim || d_out > kMaxDim) return GM_ERR_SHAPE;
  if (d_in % 8 || d_out % 8) return GM_ERR_SHAPE;
  if (!group_shape_ok(g, g_out)) return GM_ERR_SHAPE;
  if (d_in % list_width(g) || d_out % g_out) return GM_ERR_SHAPE;
  if (d_in / unit_width(g) > kMaxUnits) return GM_ERR_SHAPE;
  // The GEMMs address every matrix with 32-bit byte offsets below 2 GiB.
  const int64_t t8 = (T + 7) / 8 * 8;
  if (t8 * d_in > kMaxElems || t8 * d_out > kMaxElems || d_out * d_in > kMaxElems) return GM_ERR_SHAPE;
  return GM_OK;
}

// Split K of the forward GEMM: a launch of 256 x 256 tiles with at most 128
// tiles (half the CUs or fewer, e.g. T = 512 at LLaMA-2-13B shapes) spreads
// each tile's K range over ksplit blocks, up to 256 blocks in all, at most 8
// shares and at least four column units per share (fewer, longer shares
// measured 3.6 % faster per LLaMA-2-13B layer at T = 512 than two-unit ones);
// launches of at most 16 tiles (the 128-token, 1024 x 1024 linear has 4) may
// take shares of a single unit, since there the latency of one long K range,
// not the per-share cost, sets the time.  The partial tiles take
// ksplit * T * d_out fp32 of workspace.
constexpr int64_t kSplitMaxTiles = 128, kSplitBlocks = 256, kSplitMax = 8, kSplitFewTiles = 16;

int fwd_splits(int64_t T, int64_t d_in, int64_t d_out, int32_t g) {
  if (T <= kDecodeTokens) return 1;
  const int64_t tiles = ((T + 255) / 256) * ((d_out + 255) / 256);
  if (tiles > kSplitMaxTiles) return 1;
  int64_t ks = kSplitBlocks / tiles;
  ks = std::min(ks, kSplitMax);
  ks = std::min(ks, d_in / unit_width(g) / (tiles <= kSplitFewTiles ? 1 : 4));
  return int(std::max<int64_t>(ks, 1));
}

size_t fwd_workspace(int64_t T, int64_t d_in, int64_t d_out, int32_t g) {
  const int ks = fwd_splits(T, d_in, d_out, g);
  return ks > 1 ? round_up(size_t(ks) * size_t(T) * size_t(d_out) * sizeof(float), 256) : 0;
}

// Workspace of the backward, each part 256-byte aligned, over NL = d_in / lc
// list columns of lc = max(g, 64) input columns (nsub = lc / g groups each):
//   colcount [NL] int32 | colsoft [NL] int32 | rows [NL * d_out + 128] int32 |
//   scales [(NL * d_out + 128) * nsub] fp32 | subbits [NL * d_out + 128] int32 (nsub > 1) |
//   dYt [d_out * ldt] bf16
// The 128 spare entries after the column lists keep the dX kernel's look-ahead
// reads of the list (up to 63 entries past a column's end) inside the buffer.
struct BwdLayout {
  size_t colcount, colsoft, rows, scales, subbits, dyt, total;
  int ldt, nsub;
};

BwdLayout bwd_layout(int64_t T, int64_t d_in, int64_t d_out, int32_t g) {
  BwdLayout L;
  L.nsub = int(list_width(g) / g);
  const size_t NL = size_t(d_in / list_width(g));
  const size_t list = NL * size_t(d_out) + 128;
  L.ldt = int(round_up(size_t(T), 8));
  size_t off = 0;
  L.colcount = off;
  off = round_up(off + NL * sizeof(int32_t), 256);
  L.colsoft = off;
  off = round_up(off + NL * sizeof(int32_t), 256);
  L.rows = off;
  off = round_up(off + list * sizeof(int32_t), 256);
  L.scales = off;
  off = round_up(off + list * size_t(L.nsub) * sizeof(float), 256);
  L.subbits = off;
  if (L.nsub > 1) off = round_up(off + list * sizeof(int32_t), 256);
  L.dyt = off;
  off = round_up(off + size_t(d_out) * size_t(L.ldt) * sizeof(uint16_t), 256);
  L.total = off;
  return L;
}

// Distillation loss: limits keep every 32-bit byte offset of its GEMMs below 2^31.
constexpr int64_t kMaxHidden = 65536;
constexpr int64_t kMaxVocab = int64_t(1) << 20;

gm_status check_distill_shape(int64_t N, int64_t d, int64_t V) {
  if (N < 1 || d < 32 || V < 8) return GM_ERR_SHAPE;
  if (N > kMaxDim || d > kMaxHidden || V > kMaxVocab) return GM_ERR_SHAPE;
  if (d % 32 || V % 8) return GM_ERR_SHAPE;
  const int64_t ldv = (V + 31) / 32 * 32;
  if (V * d > kMaxElems || N * d > kMaxElems || N * ldv > kMaxElems) return GM_ERR_SHAPE;
  return GM_OK;
}

// Workspace of the distillation loss, each part 256-byte aligned:
//   z_T, z_S [N, V] fp32 | statistics [N, ceil(V/256), 5] fp32 |
//   lse_T, lse_S, cross-entropy, token weight [N] fp32 each | dz_S [N, ldv] bf16
struct DistillLayout {
  size_t zt, zs, part, lse_t, lse_s, ce, wtok, dz, total;
  int ldv, tiles;
};

DistillLayout distill_layout(int64_t N, int64_t V) {
  DistillLayout L;
  L.ldv = int((V + 31) / 32 * 32);
  L.tiles = gm::distill_vocab_tiles(int(V));
  const size_t n = size_t(N);
  size_t off = 0;
  auto take = [&](size_t& at, size_t bytes) {
    at = off;
    off = round_up(off + bytes, 256);
  };
  take(L.zt, n * size_t(V) * 4);
  take(L.zs, n * size_t(V) * 4);
  take(L.part, 5 * size_t(L.tiles) * n * 4);
  take(L.lse_t, n * 4);
  take(L.lse_s, n * 4);
  take(L.ce, n * 4);
  take(L.wtok, n * 4);
  take(L.dz, n * size_t(L.ldv) * 2);
  L.total = off;
  return L;
}

// Hypernetwork sizes.
constexpr int64_t kMaxLayers = 65536;
constexpr int64_t kMaxZ = 4096;

gm_status check_hyper_shape(int64_t L, int64_t D, int64_t H, int64_t G_total) {
  if (L < 1 || L > kMaxLayers || D < 1 || D > kMaxZ) return GM_ERR_SHAPE;
  if (H != 32 && H != 64 && H != 128) return GM_ERR_SHAPE;
  if (G_total < 1 || G_total > (int64_t(1) << 40) / (2 * H)) return GM_ERR_SHAPE;
  if (G_total / 2048 + L > int64_t(1) << 30) return GM_ERR_SHAPE;
  return GM_OK;
}

gm_status check_adamw(double lr, double beta1, double beta2, double eps, double wd, int32_t step) {
  if (!(std::isfinite(lr) && lr >= 0.0)) return GM_ERR_VALUE;
  if (!(beta1 >= 0.0 && beta1 < 1.0 && beta2 >= 0.0 && beta2 < 1.0)) return GM_ERR_VALUE;
  if (!(std::isfinite(eps) && eps > 0.0)) return GM_ERR_VALUE;
  if (!(std::isfinite(wd) && wd >= 0.0)) return GM_ERR_VALUE;
  if (step < 1) return GM_ERR_VALUE;
  return GM_OK;
}

// Workspace of the hypernetwork calls, each part 256-byte aligned (see gm::HyperWs).
struct HyperLayout {
  size_t gi, cache, o, lay, start, end, first, count, part, dout, dgi, dgh, total;
};

HyperLayout hyper_layout(int64_t L, int64_t H, int64_t G_total) {
  HyperLayout Y;
  const size_t l = size_t(L), h = size_t(H), mc = size_t(gm::hyper_max_chunks(G_total, int(L)));
  size_t off = 0;
  auto take = [&](size_t& at, size_t bytes) {
    at = off;
    off = round_up(off + bytes, 256);
  };
  take(Y.gi, 2 * l * 3 * h * 4);
  take(Y.cache, 2 * l * 5 * h * 4);
  take(Y.o, l * 2 * h * 4);
  take(Y.lay, mc * 4);
  take(Y.start, mc * 8);
  take(Y.end, mc * 8);
  take(Y.first, (l + 1) * 4);
  take(Y.count, 4);
  take(Y.part, mc * 2 * h * 4);
  take(Y.dout, l * 2 * h * 4);
  take(Y.dgi, 2 * l * 3 * h * 4);
  take(Y.dgh, 2 * l * 3 * h * 4);
  Y.total = off;
  return Y;
}

gm::HyperWs hyper_ws(void* ws, const HyperLayout& Y) {
  char* b = static_cast<char*>(ws);
  gm::HyperWs w;
  w.gi = reinterpret_cast<float*>(b + Y.gi);
  w.cache = reinterpret_cast<float*>(b + Y.cache);
  w.o = reinterpret_cast<float*>(b + Y.o);
  w.lay = reinterpret_cast<int*>(b + Y.lay);
  w.start = reinterpret_cast<int64_t*>(b + Y.start);
  w.end = reinterpret_cast<int64_t*>(b + Y.end);
  w.first = reinterpret_cast<int*>(b + Y.first);
  w.count = reinterpret_cast<int*>(b + Y.count);
  w.part = reinterpret_cast<float*>(b + Y.part);
  w.dout = reinterpret_cast<float*>(b + Y.dout);
  w.dgi = reinterpret_cast<float*>(b + Y.dgi);
  w.dgh = reinterpret_cast<float*>(b + Y.dgh);
  return w;
}

}  // namespace

GM_EXPORT int gm_abi_version(void) { return GM_ABI_VERSION; }

GM_EXPORT const char* gm_status_string(gm_status status) {
  switch (status) {
    case GM_OK: return "ok";
    case GM_ERR_NULL: return "a required pointer is NULL";
    case GM_ERR_SHAPE: return "a size is out of range or inconsistent";
    case GM_ERR_VALUE: return "a scalar argument is out of range";
    case GM_ERR_ALIGN: return "a pointer is not 16-byte aligned";
    case GM_ERR_WORKSPACE: return "workspace missing or too small";
    case GM_ERR_DEVICE: return "unsupported device or HIP launch error";
  }
  return "unknown status";
}

GM_EXPORT gm_status gm_gate(const float* logits, const float* noise, int64_t n, float tau, int hard,
                            float* mask_out, float* soft_out, gm_stream_t stream) {
  if (!logits || !mask_out) return GM_ERR_NULL;
  if (n < 0) return GM_ERR_SHAPE;
  if (gm_status st = check_tau(tau)) return st;
  if (hard != 0 && hard != 1) return GM_ERR_VALUE;
  if (!aligned16(logits) || !aligned16(mask_out) || (noise && !aligned16(noise)) ||
      (soft_out && !aligned16(soft_out)))
    return GM_ERR_ALIGN;
  if (n == 0) return GM_OK;
  if (gm_status st = check_device()) return st;
  return from_hip(gm::launch_gate_fwd(logits, noise, n, tau, hard, mask_out, soft_out, stream));
}

GM_EXPORT gm_status gm_gate_bwd(const float* dmask, const float* soft, int64_t n, float tau, float* dlogits,
                                gm_stream_t stream) {
  if (!dmask || !soft || !dlogits) return GM_ERR_NULL;
  if (n < 0) return GM_ERR_SHAPE;
  if (gm_status st = check_tau(tau)) return st;
  if (!aligned16(dmask) || !aligned16(soft) || !aligned16(dlogits)) return GM_ERR_ALIGN;
  if (n == 0) return GM_OK;
  if (gm_status st = check_device()) return st;
  return from_hip(gm::launch_gate_bwd(dmask, soft, n, tau, dlogits, stream));
}

GM_EXPORT gm_status gm_budget_loss(const float* mask, int64_t n, const int64_t* offsets, const int64_t* params,
                                   int32_t L, float s_target, float lambda, int uniform, uint64_t* kept, double* loss,
                                   float* coeff, gm_stream_t stream) {
  if (!mask || !offsets || !params || !kept || !loss || !coeff) return GM_ERR_NULL;
  if (n < 1 || L < 1) return GM_ERR_SHAPE;
  if (!(std::isfinite(s_target) && s_target > 0.0f && s_target < 1.0f)) return GM_ERR_VALUE;
  if (!(std::isfinite(lambda) && lambda >= 0.0f)) return GM_ERR_VALUE;
  if (uniform != 0 && uniform != 1) return GM_ERR_VALUE;
  if (!aligned16(mask) || !aligned8(offsets) || !aligned8(params) || !aligned8(kept) || !aligned8(loss) ||
      !aligned4(coeff))
    return GM_ERR_ALIGN;
  if (gm_status st = check_device()) return st;
  return from_hip(gm::launch_budget_loss(mask, n, offsets, params, L, s_target, lambda, uniform,
                                         reinterpret_cast<unsigned long long*>(kept), loss, coeff, stream));
}

GM_EXPORT gm_status gm_gate_bwd_budget(const float* dgate, const float* soft, int64_t n, float tau,
                                       const int64_t* offsets, int32_t L, const float* coeff, float* dlogits,
                                       gm_stream_t stream) {
  if (!dgate || !soft || !offsets || !coeff || !dlogits) return GM_ERR_NULL;
  if (n < 1 || L < 1) return GM_ERR_SHAPE;
  if (gm_status st = check_tau(tau)) return st;
  if (!aligned16(dgate) || !aligned16(soft) || !aligned16(dlogits) || !aligned8(offsets) || !aligned4(coeff))
    return GM_ERR_ALIGN;
  if (gm_status st = check_device()) return st;
  return from_hip(gm::launch_gate_bwd_budget(dgate, soft, n, tau, offsets, L, coeff, dlogits, stream));
}

GM_EXPORT gm_status gm_workspace_size(int op, int64_t T, int64_t d_in, int64_t d_out, int32_t g, int32_t g_out,
                                      size_t* bytes) {
  if (!bytes) return GM_ERR_NULL;
  if (op != GM_OP_FWD && op != GM_OP_BWD) return GM_ERR_VALUE;
  if (gm_status st = check_linear_shape(T, d_in, d_out, g, g_out)) return st;
  *bytes = op == GM_OP_FWD ? fwd_workspace(T, d_in, d_out, g) : bwd_layout(T, d_in, d_out, g).total;
  return GM_OK;
}

GM_EXPORT gm_status gm_masked_linear_fwd(const uint16_t* X, const uint16_t* W, const float* mask, int64_t T,
                                         int64_t d_in, int64_t d_out, int32_t g, int32_t g_out, uint16_t* Y,
                                         void* ws, size_t ws_bytes, gm_stream_t stream) {
  if (!X || !W || !mask || !Y) return GM_ERR_NULL;
  if (gm_status st = check_linear_shape(T, d_in, d_out, g, g_out)) return st;
  if (!aligned16(X) || !aligned16(W) || !aligned16(mask) || !aligned16(Y) || (ws && !aligned16(ws)))
    return GM_ERR_ALIGN;
  const size_t need = fwd_workspace(T, d_in, d_out, g);
  if (ws && ws_bytes < need) return GM_ERR_WORKSPACE;
  if (gm_status st = check_device()) return st;
  const int t = int(T), di = int(d_in), dout = int(d_out);
  if (T <= kDecodeTokens && d_in / g <= gm::gemv_max_groups_per_row())
    return from_hip(gm::launch_gemv_inplace(X, W, mask, t, di, dout, g, g_out, Y, stream));
  // Without a workspace the forward runs unsplit (the same Y up to fp32 summation order).
  const int ks = ws && need ? fwd_splits(T, d_in, d_out, g) : 1;
  return from_hip(gm::launch_fwd(X, W, mask, t, di, dout, g, g_out, Y, ks, static_cast<float*>(ws), stream));
}

namespace {

// The backward after argument validation: column lists, dgate (with the dY^T
// side output when dX is wanted), dX.  `ws` holds at least bwd_layout().total
// bytes when dX is wanted.
gm_status masked_linear_bwd_launch(const uint16_t* dY, const uint16_t* X, const uint16_t* W, const float* mask,
                                   int64_t T, int64_t d_in, int64_t d_out, int32_t g, int32_t g_out, uint16_t* dX,
                                   float* dgate, void* ws, gm_stream_t stream) {
  const BwdLayout L = bwd_layout(T, d_in, d_out, g);
  const int t = int(T), di = int(d_in), dout = int(d_out), G_in = int(d_in / g);
  char* base = static_cast<char*>(ws);
  uint16_t* dyt = dX ? reinterpret_cast<uint16_t*>(base + L.dyt) : nullptr;
  if (dX) {
    int* colcount = reinterpret_cast<int*>(base + L.colcount);
    int* colsoft = reinterpret_cast<int*>(base + L.colsoft);
    int* rows = reinterpret_cast<int*>(base + L.rows);
    float* scales = reinterpret_cast<float*>(base + L.scales);
    int* subbits = L.nsub > 1 ? reinterpret_cast<int*>(base + L.subbits) : nullptr;
    // dY^T: a side output of the dgate GEMM, whose launch also builds the
    // column lists; without dgate, a lists pass and a transpose pass.
    if (dgate) {
      if (gm_status st = from_hip(gm::launch_dgate(dY, X, W, t, di, dout, g, g_out, dgate, dyt, L.ldt, mask, L.nsub,
                                                   colcount, colsoft, rows, scales, subbits, stream)))
        return st;
    } else {
      if (gm_status st = from_hip(gm::launch_col_lists(mask, dout, G_in, g_out, L.nsub, colcount, colsoft, rows,
                                                       scales, subbits, stream)))
        return st;
      if (gm_status st = from_hip(gm::launch_transpose(dY, t, dout, dyt, L.ldt, stream))) return st;
    }
    return from_hip(gm::launch_dx(dyt, L.ldt, W, colcount, rows, scales, subbits, colsoft, t, di, dout, g, dX,
                                  stream));
  }
  return from_hip(gm::launch_dgate(dY, X, W, t, di, dout, g, g_out, dgate, nullptr, 0, nullptr, 1, nullptr, nullptr,
                                   nullptr, nullptr, nullptr, stream));
}

// Shared argument checks of the two backward entry points (everything but the workspace).
gm_status check_bwd_args(const uint16_t* dY, const uint16_t* X, const uint16_t* W, const float* mask, int64_t T,
                         int64_t d_in, int64_t d_out, int32_t g, int32_t g_out, const uint16_t* dX,
                         const float* dgate) {
  if (!dY || !X || !W) return GM_ERR_NULL;
  if (dX && !mask) return GM_ERR_NULL;
  if (gm_status st = check_linear_shape(T, d_in, d_out, g, g_out)) return st;
  if (!aligned16(dY) || !aligned16(X) || !aligned16(W) || (mask && !aligned16(mask)) || (dX && !aligned16(dX)) ||
      (dgate && !aligned16(dgate)))
    return GM_ERR_ALIGN;
  return GM_OK;
}

// Scratch of the allocation-free backward: a file-scope device array that
// every device the library runs on holds until the process ends.  In host
// code `scratch` names a host-side stand-in, never the device memory: its
// device address is looked up once per device (with that device current) and
// only that address is handed to kernels.
constexpr size_t kNoAllocScratchBytes = GM_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

gm_status noalloc_scratch(void** out) {
  static std::mutex mu;
  static void* ptr[256];
  int dev = 0;
  if (hipError_t e = hipGetDevice(&dev)) return device_error("hipGetDevice", e);
  if (dev < 0 || dev >= 256) return device_error("device index", hipErrorInvalidDevice);
  std::lock_guard<std::mutex> lock(mu);
  if (ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) return device_error("hipGetSymbolAddress", e);
    if (p == nullptr || !aligned16(p)) return device_error("scratch address", hipErrorInvalidValue);
    ptr[dev] = p;
  }
  *out = ptr[dev];
  return GM_OK;
}

}  // namespace

GM_EXPORT gm_status gm_masked_linear_bwd(const uint16_t* dY, const uint16_t* X, const uint16_t* W,
                                         const float* mask, int64_t T, int64_t d_in, int64_t d_out, int32_t g,
                                         int32_t g_out, uint16_t* dX, float* dgate, void* ws, size_t ws_bytes,
                                         gm_stream_t stream) {
  if (gm_status st = check_bwd_args(dY, X, W, mask, T, d_in, d_out, g, g_out, dX, dgate)) return st;
  if (!dX && !dgate) return GM_OK;
  if (dX) {
    if (!ws) return GM_ERR_WORKSPACE;
    if (ws_bytes < bwd_layout(T, d_in, d_out, g).total) return GM_ERR_WORKSPACE;
    if (!aligned16(ws)) return GM_ERR_ALIGN;
  }
  if (gm_status st = check_device()) return st;
  return masked_linear_bwd_launch(dY, X, W, mask, T, d_in, d_out, g, g_out, dX, dgate, ws, stream);
}

GM_EXPORT gm_status gm_masked_linear_bwd_noalloc(const uint16_t* dY, const uint16_t* X, const uint16_t* W,
                                                 const float* mask, int64_t T, int64_t d_in, int64_t d_out,
                                                 int32_t g, int32_t g_out, uint16_t* dX, float* dgate,
                                                 gm_stream_t stream) {
  if (gm_status st = check_bwd_args(dY, X, W, mask, T, d_in, d_out, g, g_out, dX, dgate)) return st;
  if (!dX && !dgate) return GM_OK;
  if (dX && bwd_layout(T, d_in, d_out, g).total > kNoAllocScratchBytes) return GM_ERR_WORKSPACE;
  if (gm_status st = check_device()) return st;
  void* ws = nullptr;
  if (dX)
    if (gm_status st = noalloc_scratch(&ws)) return st;
  return masked_linear_bwd_launch(dY, X, W, mask, T, d_in, d_out, g, g_out, dX, dgate, ws, stream);
}

GM_EXPORT gm_status gm_pack_rows(const uint16_t* W, const float* mask, int64_t d_in, int64_t d_out, int32_t g,
                                 int32_t g_out, int64_t capacity, uint16_t* Wp, int32_t* chunk, float* scale,
                                 int32_t* rowptr, gm_stream_t stream) {
  if (!W || !mask || !Wp || !chunk || !scale || !rowptr) return GM_ERR_NULL;
  if (gm_status st = check_linear_shape(1, d_in, d_out, g, g_out)) return st;
  if (capacity < 0 || capacity > d_out * (d_in / g)) return GM_ERR_SHAPE;
  if (!aligned16(W) || !aligned16(mask) || !aligned16(Wp) || !aligned16(chunk) || !aligned16(scale) ||
      !aligned16(rowptr))
    return GM_ERR_ALIGN;
  if (gm_status st = check_device()) return st;
  return from_hip(gm::launch_pack_rows(W, mask, int(d_in), int(d_out), g, g_out, capacity, Wp, chunk, scale,
                                       rowptr, stream));
}

GM_EXPORT gm_status gm_packed_linear_fwd(const uint16_t* X, const uint16_t* Wp, const int32_t* chunk,
                                         const float* scale, const int32_t* rowptr, int64_t T, int64_t d_in,
                                         int64_t d_out, int32_t g, uint16_t* Y, gm_stream_t stream) {
  if (!X || !Wp || !chunk || !scale || !rowptr || !Y) return GM_ERR_NULL;
  // the export holds row pieces of g weights whatever the group's height
  if (gm_status st = check_linear_shape(T, d_in, d_out, g, g < 64 ? g : 1)) return st;
  if (!aligned16(X) || !aligned16(Wp) || !aligned16(chunk) || !aligned16(scale) || !aligned16(rowptr) ||
      !aligned16(Y))
    return GM_ERR_ALIGN;
  if (gm_status st = check_device()) return st;
  return from_hip(
      gm::launch_gemv_packed(X, Wp, chunk, scale, rowptr, int(T), int(d_in), int(d_out), g, Y, stream));
}

GM_EXPORT gm_status gm_distill_workspace_size(int64_t N, int64_t d, int64_t V, size_t* bytes) {
  if (!bytes) return GM_ERR_NULL;
  if (gm_status st = check_distill_shape(N, d, V)) return st;
  *bytes = distill_layout(N, V).total;
  return GM_OK;
}

GM_EXPORT gm_status gm_distill_fwd(const uint16_t* Ht, const uint16_t* Hs, const uint16_t* W, const uint8_t* valid,
                                   int64_t N, int64_t d, int64_t V, float* loss, float* ce, void* ws,
                                   size_t ws_bytes, gm_stream_t stream) {
  if (!Ht || !Hs || !W || !loss || !ws) return GM_ERR_NULL;
  if (gm_status st = check_distill_shape(N, d, V)) return st;
  if (!aligned16(Ht) || !aligned16(Hs) || !aligned16(W) || !aligned16(ws) || !aligned4(loss) || (ce && !aligned4(ce)))
    return GM_ERR_ALIGN;
  const DistillLayout L = distill_layout(N, V);
  if (ws_bytes < L.total) return GM_ERR_WORKSPACE;
  if (gm_status st = check_device()) return st;
  char* b = static_cast<char*>(ws);
  auto f = [&](size_t off) { return reinterpret_cast<float*>(b + off); };
  return from_hip(gm::launch_distill_fwd(Ht, Hs, W, valid, int(N), int(d), int(V), f(L.zt), f(L.zs), f(L.part),
                                         f(L.lse_t), f(L.lse_s), f(L.ce), f(L.wtok), loss, ce, stream));
}

GM_EXPORT gm_status gm_distill_bwd(const uint16_t* W, int64_t N, int64_t d, int64_t V, uint16_t* dHs, void* ws,
                                   size_t ws_bytes, gm_stream_t stream) {
  if (!W || !dHs || !ws) return GM_ERR_NULL;
  if (gm_status st = check_distill_shape(N, d, V)) return st;
  if (!aligned16(W) || !aligned16(dHs) || !aligned16(ws)) return GM_ERR_ALIGN;
  const DistillLayout L = distill_layout(N, V);
  if (ws_bytes < L.total) return GM_ERR_WORKSPACE;
  if (gm_status st = check_device()) return st;
  char* b = static_cast<char*>(ws);
  auto f = [&](size_t off) { return reinterpret_cast<float*>(b + off); };
  return from_hip(gm::launch_distill_bwd(W, int(N), int(d), int(V), f(L.zt), f(L.zs), f(L.lse_t), f(L.lse_s),
                                         f(L.wtok), reinterpret_cast<uint16_t*>(b + L.dz), L.ldv, dHs, stream));
}

GM_EXPORT gm_status gm_hyper_workspace_size(int64_t L, int64_t D, int64_t H, int64_t G_total, size_t* bytes) {
  if (!bytes) return GM_ERR_NULL;
  if (gm_status st = check_hyper_shape(L, D, H, G_total)) return st;
  *bytes = hyper_layout(L, H, G_total).total;
  return GM_OK;
}

GM_EXPORT gm_status gm_hyper_fwd(const float* z, const float* gru, const float* A, const float* c,
                                 const int64_t* offsets, int64_t L, int64_t D, int64_t H, int64_t G_total,
                                 float* logits, void* ws, size_t ws_bytes, gm_stream_t stream) {
  if (!z || !gru || !A || !c || !offsets || !logits || !ws) return GM_ERR_NULL;
  if (gm_status st = check_hyper_shape(L, D, H, G_total)) return st;
  if (!aligned4(z) || !aligned4(gru) || !aligned16(A) || !aligned4(c) || !aligned8(offsets) || !aligned4(logits) ||
      !aligned16(ws))
    return GM_ERR_ALIGN;
  const HyperLayout Y = hyper_layout(L, H, G_total);
  if (ws_bytes < Y.total) return GM_ERR_WORKSPACE;
  if (gm_status st = check_device()) return st;
  return from_hip(gm::launch_hyper_fwd(z, gru, A, c, offsets, int(L), int(D), int(H), G_total, logits,
                                       hyper_ws(ws, Y), stream));
}

GM_EXPORT gm_status gm_hyper_bwd(const float* dlogits, const float* z, const float* gru, float* A, float* c,
                                 float* mA, float* vA, float* mc, float* vc, int64_t L, int64_t D, int64_t H,
                                 int64_t G_total, double lr, double beta1, double beta2, double eps,
                                 double weight_decay, int32_t step, float* dgru, void* ws, size_t ws_bytes,
                                 gm_stream_t stream) {
  if (!dlogits || !z || !gru || !A || !c || !mA || !vA || !mc || !vc || !dgru || !ws) return GM_ERR_NULL;
  if (gm_status st = check_hyper_shape(L, D, H, G_total)) return st;
  if (gm_status st = check_adamw(lr, beta1, beta2, eps, weight_decay, step)) return st;
  if (!aligned4(dlogits) || !aligned4(z) || !aligned4(gru) || !aligned16(A) || !aligned4(c) || !aligned16(mA) ||
      !aligned16(vA) || !aligned4(mc) || !aligned4(vc) || !aligned4(dgru) || !aligned16(ws))
    return GM_ERR_ALIGN;
  const HyperLayout Y = hyper_layout(L, H, G_total);
  if (ws_bytes < Y.total) return GM_ERR_WORKSPACE;
  if (gm_status st = check_device()) return st;
  return from_hip(gm::launch_hyper_bwd(dlogits, z, gru, A, c, mA, vA, mc, vc, int(L), int(D), int(H), G_total, lr,
                                       beta1, beta2, eps, weight_decay, step, dgru, hyper_ws(ws, Y), stream));
}

GM_EXPORT gm_status gm_adamw(float* p, const float* g, float* m, float* v, int64_t n, double lr, double beta1,
                             double beta2, double eps, double weight_decay, int32_t step, gm_stream_t stream) {
  if (!p || !g || !m || !v) return GM_ERR_NULL;
  if (n < 0) return GM_ERR_SHAPE;
  if (gm_status st = check_adamw(lr, beta1, beta2, eps, weight_decay, step)) return st;
  if (!aligned4(p) || !aligned4(g) || !aligned4(m) || !aligned4(v)) return GM_ERR_ALIGN;
  if (n == 0) return GM_OK;
  if (gm_status st = check_device()) return st;
  return from_hip(gm::launch_adamw(p, g, m, v, n, lr, beta1, beta2, eps, weight_decay, step, stream));
}
