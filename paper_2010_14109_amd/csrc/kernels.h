// Host-side launchers of the HIP kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include "internal.h"

namespace ooc {

// Runs function fn on stream s; ptrs[j] is the device address of fn.vars[j],
// bytes[j] its size.
hipError_t launch_fn(const Fn& fn, void* const* ptrs, const uint64_t* bytes, float lr, float mu,
                     hipStream_t s);

// GEMM family (gemm.hip).  Shapes as in the operation table of ooc.h.
hipError_t linear_fwd(const float* X, const float* W, const float* b, float* Y, int64_t M,
                      int64_t K, int64_t N, hipStream_t s);
hipError_t linear_bwd_w(const float* X, const float* dY, float* dW, float* db, float* part,
                        int64_t slices, int64_t M, int64_t K, int64_t N, hipStream_t s);
hipError_t linear_bwd_x(const float* W, const float* dY, float* dX, int64_t M, int64_t K,
                        int64_t N, hipStream_t s);
// Batched GEMM: C_z[M][N] = sum_k A_z[m][k] B_z[k][n] for z < batches.  A is
// "row of k" (A[m][k] = A[m lda + k]) or not (A[m][k] = A[k lda + m]); B is
// "row of k" (B[k][n] = B[n ldb + k]) or not (B[k][n] = B[k ldb + n]).
// Batch z = zo inner + zi moves A, B, C by zo * outer + zi * inner strides.
struct BatchStrides {
  int64_t inner;
  int64_t a_outer, a_inner, b_outer, b_inner, c_outer, c_inner;
  // nonzero: C tiles whose every entry lies above the diagonal (column > row) are left unwritten
  int64_t skip_upper = 0;
};
hipError_t gemm_batched(bool a_rowk, const float* A, int64_t lda, bool b_rowk, const float* B,
                        int64_t ldb, float* C, int64_t ldc, int64_t M, int64_t N, int64_t K,
                        int64_t batches, const BatchStrides& st, hipStream_t s);

struct ConvShape {
  int64_t N, H, W, C, K, R, S, stride, pad, P, Q;
};
hipError_t conv_fwd(const float* X, const float* W, float* Y, const ConvShape& c, hipStream_t s);
hipError_t conv_bwd_x(const float* W, const float* dY, float* dX, const ConvShape& c,
                      hipStream_t s);
hipError_t conv_bwd_w(const float* X, const float* dY, float* dW, float* part, int64_t slices,
                      const ConvShape& c, hipStream_t s);
// Split-K slice count the weight-gradient launchers run best with: M x N
// outputs reduced over K rows; C = input channels of a filter gradient, -1 for
// a dense layer.
int64_t wgrad_slices(int64_t M, int64_t N, int64_t K, int64_t C);

// Elementwise, loss, update, normalisation and pooling (ops.hip).
hipError_t relu_fwd(const float* x, float* y, int64_t n, hipStream_t s);
hipError_t relu_bwd(const float* y, const float* dy, float* dx, int64_t n, hipStream_t s);
hipError_t add(const float* a, const float* b, float* y, int64_t n, hipStream_t s);
// a += b in place (a and b distinct)
hipError_t accumulate(float* a, const float* b, int64_t n, hipStream_t s);
// count parameter tensors: w[k] -= lr * (v[k] = mu v[k] + g[k]), or lr * g[k] where v[k] is null
hipError_t sgd(int count, float* const* w, const float* const* g, float* const* v,
               const int64_t* n, float lr, float mu, hipStream_t s);
hipError_t softmax_ce(const float* logits, const int32_t* labels, float* loss, float* dlogits,
                      int64_t N, int64_t classes, hipStream_t s);
hipError_t bn_fwd(const float* x, const float* gamma, const float* beta, float* y, float* stats,
                  int64_t rows, int64_t C, int64_t slices, hipStream_t s);
hipError_t bn_bwd(const float* x, const float* gamma, float* stats, const float* dy, float* dx,
                  float* dgamma, float* dbeta, int64_t rows, int64_t C, int64_t slices,
                  hipStream_t s);
struct PoolShape {
  int64_t N, H, W, C, k, stride, pad, P, Q;
};
hipError_t maxpool_fwd(const float* x, float* y, uint8_t* idx, const PoolShape& p, hipStream_t s);
hipError_t maxpool_bwd(const uint8_t* idx, const float* dy, float* dx, const PoolShape& p,
                       hipStream_t s);
// Channel concatenation (forward: parts -> cat; backward: cat -> parts) and
// nearest 2x upsampling (forward: in [N H W C] -> out; backward: the gradient
// of out -> in [N H W C]).
hipError_t concat(bool forward, float* cat, void* const* parts, const int64_t* cs, int k,
                  int64_t rows, hipStream_t s);
hipError_t upsample(bool forward, const float* in, float* out, int64_t N, int64_t H, int64_t W,
                    int64_t C, hipStream_t s);
hipError_t avgpool_fwd(const float* x, float* y, int64_t N, int64_t HW, int64_t C, hipStream_t s);
hipError_t avgpool_bwd(const float* dy, float* dx, int64_t N, int64_t HW, int64_t C,
                       hipStream_t s);
// Transformer layers (transformer.hip).
hipError_t embed_fwd(const int32_t* ids, const float* E, const float* pos, float* y, int64_t B,
                     int64_t T, int64_t V, int64_t d, hipStream_t s);
hipError_t embed_bwd(const int32_t* ids, const float* dy, float* dE, float* dpos, int64_t B,
                     int64_t T, int64_t V, int64_t d, hipStream_t s);
hipError_t layernorm_fwd(const float* x, const float* gamma, const float* beta, float* y,
                         float* stats, int64_t rows, int64_t d, int64_t slices, hipStream_t s);
hipError_t layernorm_bwd(const float* x, const float* gamma, float* stats, const float* dy,
                         float* dx, float* dgamma, float* dbeta, int64_t rows, int64_t d,
                         int64_t slices, hipStream_t s);
hipError_t gelu_fwd(const float* x, float* y, int64_t n, hipStream_t s);
hipError_t gelu_bwd(const float* x, const float* dy, float* dx, int64_t n, hipStream_t s);
hipError_t attention_fwd(const float* qkv, float* P, float* y, int64_t B, int64_t T, int64_t H,
                         int64_t dh, bool causal, hipStream_t s);
hipError_t attention_bwd(const float* qkv, float* P, const float* dy, float* dqkv, float* dS,
                         int64_t B, int64_t T, int64_t H, int64_t dh, bool causal, hipStream_t s);

hipError_t mix(void* const* ptrs, const uint64_t* words, int nvars, uint32_t seed, hipStream_t s,
               bool y_read);

}  // namespace ooc
