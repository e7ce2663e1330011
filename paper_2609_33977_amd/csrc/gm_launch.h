// Host-side launchers of the gfx950 kernels (internal to the library).
// Every launcher enqueues on stream s and returns the launch status; argument
// validation happens in the C-ABI layer before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gm {

hipError_t launch_gate_fwd(const float* logits, const float* noise, int64_t n, float tau, int hard, float* mask,
                           float* soft, hipStream_t s);
hipError_t launch_gate_bwd(const float* dmask, const float* soft, int64_t n, float tau, float* dlogits,
                           hipStream_t s);

hipError_t launch_budget_loss(const float* mask, int64_t n, const int64_t* offsets, const int64_t* params, int L,
                              float s_target, float lambda, int uniform, unsigned long long* kept, double* loss,
                              float* coeff, hipStream_t s);
hipError_t launch_gate_bwd_budget(const float* dgate, const float* soft, int64_t n, float tau,
                                  const int64_t* offsets, int L, const float* coeff, float* dlogits, hipStream_t s);

// Group shapes: g_out x g (go = g_out; 1 for row groups).
hipError_t launch_col_lists(const float* mask, int d_out, int G_in, int go, int nsub, int* colcount, int* colsoft,
                            int* rows, float* scales, int* subbits, hipStream_t s);
hipError_t launch_pack_rows(const uint16_t* W, const float* mask, int d_in, int d_out, int g, int go,
                            int64_t capacity, uint16_t* Wp, int* chunk, float* scale, int* rowptr, hipStream_t s);

hipError_t launch_gemv_inplace(const uint16_t* X, const uint16_t* W, const float* mask, int T, int d_in, int d_out,
                               int g, int go, uint16_t* Y, hipStream_t s);
hipError_t launch_gemv_packed(const uint16_t* X, const uint16_t* Wp, const int* chunk, const float* scale,
                              const int* rowptr, int T, int d_in, int d_out, int g, uint16_t* Y, hipStream_t s);
int gemv_max_groups_per_row();

// ksplit > 1 splits each tile's K range over that many blocks, which store fp32
// partial tiles into part [ksplit][T][d_out]; a second kernel adds them in order.
hipError_t launch_fwd(const uint16_t* X, const uint16_t* W, const float* mask, int T, int d_in, int d_out, int g,
                      int go, uint16_t* Y, int ksplit, float* part, hipStream_t s);
// With colcount set, the launch also builds the column lists (as launch_col_lists).
hipError_t launch_dgate(const uint16_t* dY, const uint16_t* X, const uint16_t* W, int T, int d_in, int d_out, int g,
                        int go, float* dgate, uint16_t* dYt, int ldt, const float* mask, int nsub, int* colcount,
                        int* colsoft, int* rows, float* scales, int* subbits, hipStream_t s);
hipError_t launch_transpose(const uint16_t* dY, int T, int d_out, uint16_t* dYt, int ldt, hipStream_t s);
hipError_t launch_dx(const uint16_t* dYt, int ldt, const uint16_t* W, const int* colcount, const int* rows,
                     const float* scales, const int* subbits, const int* colsoft, int T, int d_in, int d_out, int g,
                     uint16_t* dX, hipStream_t s);

// Distillation loss (Sec. 2.4, Eq. 4) through the LM head.
int distill_vocab_tiles(int V);
hipError_t launch_distill_fwd(const uint16_t* Ht, const uint16_t* Hs, const uint16_t* W, const uint8_t* valid, int N,
                              int d, int V, float* zt, float* zs, float* part, float* lse_t, float* lse_s, float* ce,
                              float* wtok, float* loss, float* ce_out, hipStream_t s);
hipError_t launch_distill_bwd(const uint16_t* W, int N, int d, int V, const float* zt, const float* zs,
                              const float* lse_t, const float* lse_s, const float* wtok, uint16_t* dz, int ldv,
                              uint16_t* dH, hipStream_t s);

// Hypernetwork (Sec. 2.2, Eq. 3) and AdamW.
struct HyperWs {
  float* gi;       // [2][L][3H] input part of the gates
  float* cache;    // [2][L][5H] h_prev, r, u, n, W_hn h_prev + b_hn
  float* o;        // [L][2H] GRU outputs
  int* lay;        // [max chunks] layer of each head chunk
  int64_t* start;  // [max chunks] first row
  int64_t* end;    // [max chunks] one past the last row
  int* first;      // [L + 1] first chunk of each layer
  int* count;      // [1] number of chunks
  float* part;     // [max chunks][2H] chunk partials of do
  float* dout;     // [L][2H] gradient of the GRU outputs
  float* dgi;      // [2][L][3H] gate gradients, input side
  float* dgh;      // [2][L][3H] gate gradients, recurrent side
};
int hyper_max_chunks(int64_t G_total, int L);
hipError_t launch_hyper_fwd(const float* z, const float* gru, const float* A, const float* c, const int64_t* offsets,
                            int L, int D, int H, int64_t G_total, float* logits, const HyperWs& w, hipStream_t s);
hipError_t launch_hyper_bwd(const float* dlogits, const float* z, const float* gru, float* A, float* c, float* mA,
                            float* vA, float* mc, float* vc, int L, int D, int H, int64_t G_total, double lr,
                            double beta1, double beta2, double eps, double weight_decay, int step, float* dgru,
                            const HyperWs& w, hipStream_t s);
hipError_t launch_adamw(float* p, const float* g, float* m, float* v, int64_t n, double lr, double beta1,
                        double beta2, double eps, double weight_decay, int step, hipStream_t s);

}  // namespace gm
