// Dense and convolution layers as one fp32 MFMA GEMM kernel (gfx950).
//
// C[M][N] = sum_k A[m][k] B[k][n].  A 256-thread workgroup computes a
// 128 x 128 tile of C (or 128 x 64 / 64 x 128 when one side is at most 64
// wide); each of its four wave64s owns a quarter of the tile made of
// v_mfma_f32_32x32x2f32 blocks (2 x 2 of them for 128 x 128).  K is walked in tiles of 32,
// double-buffered through LDS: while the waves multiply tile t out of one
// buffer, every thread has tile t+1 in flight from global memory into
// registers and writes it to the other buffer.  Within a K tile the two
// half-waves take the two halves of the tile (the MFMA reduces over both), so
// each lane reads four consecutive k values of its row at once.
//
// Operands reach LDS through loaders, one per way the operand sits in
// memory: plain row-major matrices (contiguous along k, or along m / n) and
// the implicit-GEMM views of NHWC convolutions (forward: the input patches;
// input gradient: the output gradient gathered through the filter taps;
// filter gradient: the input patches seen along the batch-pixel axis).  A
// loader zero-fills everything outside the matrix, so no shape needs
// padding.  LDS layout follows the contiguous direction: "row of k" tiles
// ([rows][32 + 4]) are written and read with 16-byte accesses, "row of m"
// tiles ([32][rows + 4]) are written with 16-byte accesses and read with
// 4-byte ones; the +4 pads keep half-wave reads free of bank conflicts.
//
// Split-K: the filter gradients reduce over N P Q pixels or over the rows of
// a dense layer (up to millions), so the grid's second dimension cuts that
// axis into slices whose partial tiles go to separate buffers and are summed
// afterwards in slice order.  A dense layer's bias gradient (the column sums
// of dY) is taken from the A tiles already in LDS by the workgroups of the
// first tile column, slice by slice like dW.  No atomics anywhere: results
// do not depend on scheduling or addresses.
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace ooc {

namespace {

constexpr int BK = 32;
constexpr int LDK = BK + 4;    // row-of-k tile stride (floats)
constexpr int THREADS = 256;

typedef float floatx16 __attribute__((ext_vector_type(16)));

__device__ inline float4 zero4() { return make_float4(0.f, 0.f, 0.f, 0.f); }

// ---------------------------------------------------------------- loaders
// A loader feeds one operand tile of extent E (tile rows along m or n) by 32
// along k.  init(mn0, MN) runs once per workgroup (mn0 = tile origin, MN =
// extent of the matrix), fetch(k0, kend, r) loads this thread's E / 8 values
// of the K tile starting at k0 as E / 32 float4 (zero at k >= kend),
// store(lds, r) writes them.
//
// Row-of-k layout [E][32 + 4]: thread t loads rows (t >> 3) + 32 j, k offset
// (t & 7) * 4.  Row-of-m layout [32][E + 4]: E / 4 threads per k row; thread
// t loads k rows t / (E / 4) + (1024 / E) j, m offset (t % (E / 4)) * 4.

template <int E>
struct RowK {
  static constexpr bool kRowOfK = true;
  static constexpr int kN = E / 32;
  static constexpr int kLds = E * LDK;
  __device__ static int row(int j) { return (threadIdx.x >> 3) + 32 * j; }
  __device__ static int koff() { return (threadIdx.x & 7) * 4; }
  __device__ static void store(float* lds, const float4 (&r)[kN]) {
#pragma unroll
    for (int j = 0; j < kN; ++j) *reinterpret_cast<float4*>(&lds[row(j) * LDK + koff()]) = r[j];
  }
};
template <int E>
struct RowM {
  static constexpr bool kRowOfK = false;
  static constexpr int kN = E / 32;
  static constexpr int kLd = E + 4;
  static constexpr int kLds = BK * kLd;
  __device__ static int krow(int j) { return (int)threadIdx.x / (E / 4) + (1024 / E) * j; }
  __device__ static int moff() { return ((int)threadIdx.x % (E / 4)) * 4; }
  __device__ static void store(float* lds, const float4 (&r)[kN]) {
#pragma unroll
    for (int j = 0; j < kN; ++j) *reinterpret_cast<float4*>(&lds[krow(j) * kLd + moff()]) = r[j];
  }
};

// X[i][k] = p[i * ld + k]  (contiguous along k)
template <int E, bool VEC>
struct MatK : RowK<E> {
  using Base = RowK<E>;
  const float* p;
  int64_t ld;
  int64_t row0;
  int64_t rows;
  __device__ void init(int64_t mn0, int64_t MN) {
    row0 = mn0;
    rows = MN;
  }
  __device__ void fetch(int64_t k0, int64_t kend, float4 (&r)[Base::kN]) const {
    const int64_t k = k0 + Base::koff();
#pragma unroll
    for (int j = 0; j < Base::kN; ++j) {
      const int64_t i = row0 + Base::row(j);
      const float* q = p + i * ld + k;
      if (VEC) {
        r[j] = (i < rows && k < kend) ? *reinterpret_cast<const float4*>(q) : zero4();
      } else {
        const bool ok = i < rows;
        r[j].x = (ok && k + 0 < kend) ? q[0] : 0.f;
        r[j].y = (ok && k + 1 < kend) ? q[1] : 0.f;
        r[j].z = (ok && k + 2 < kend) ? q[2] : 0.f;
        r[j].w = (ok && k + 3 < kend) ? q[3] : 0.f;
      }
    }
  }
};

// X[i][k] = p[k * ld + i]  (contiguous along m or n)
template <int E, bool VEC>
struct MatM : RowM<E> {
  using Base = RowM<E>;
  const float* p;
  int64_t ld;
  int64_t i0;
  int64_t rows;
  __device__ void init(int64_t mn0, int64_t MN) {
    i0 = mn0 + Base::moff();
    rows = MN;
  }
  __device__ void fetch(int64_t k0, int64_t kend, float4 (&r)[Base::kN]) const {
#pragma unroll
    for (int j = 0; j < Base::kN; ++j) {
      const int64_t k = k0 + Base::krow(j);
      const float* q = p + k * ld + i0;
      if (VEC) {
        r[j] = (k < kend && i0 < rows) ? *reinterpret_cast<const float4*>(q) : zero4();
      } else {
        const bool ok = k < kend;
        r[j].x = (ok && i0 + 0 < rows) ? q[0] : 0.f;
        r[j].y = (ok && i0 + 1 < rows) ? q[1] : 0.f;
        r[j].z = (ok && i0 + 2 < rows) ? q[2] : 0.f;
        r[j].w = (ok && i0 + 3 < rows) ? q[3] : 0.f;
      }
    }
  }
};

// Convolution forward, A = input patches: A[m = (n, p, q)][kk = (r, s, c)] =
// X[n][p st - pad + r][q st - pad + s][c]   (row-of-k; VEC needs C % 4 == 0)
template <int E, bool VEC>
struct ConvPatch : RowK<E> {
  using Base = RowK<E>;
  const float* x;
  int H, W, C, S, st, pad, P, Q;
  int64_t M;
  int n_[Base::kN], h_[Base::kN], w_[Base::kN];   // per row: image, top-left input coordinates
  __device__ void init(int64_t mn0, int64_t MN) {
    M = MN;
#pragma unroll
    for (int j = 0; j < Base::kN; ++j) {
      const int64_t m = mn0 + Base::row(j);
      if (m < M) {
        const int64_t pq = (int64_t)P * Q;
        const int n = (int)(m / pq);
        const int rem = (int)(m - (int64_t)n * pq);
        const int p = rem / Q, q = rem - p * Q;
        n_[j] = n;
        h_[j] = p * st - pad;
        w_[j] = q * st - pad;
      } else {
        n_[j] = -1;
      }
    }
  }
  __device__ float at(int j, int64_t kk, int64_t kend) const {
    if (n_[j] < 0 || kk >= kend) return 0.f;
    const int sc = S * C;
    const int r = (int)(kk / sc);
    const int rem = (int)(kk - (int64_t)r * sc);
    const int s = rem / C, c = rem - s * C;
    const int h = h_[j] + r, w = w_[j] + s;
    if (h < 0 || h >= H || w < 0 || w >= W) return 0.f;
    return x[(((int64_t)n_[j] * H + h) * W + w) * C + c];
  }
  __device__ void fetch(int64_t k0, int64_t kend, float4 (&r)[Base::kN]) const {
    const int64_t kk = k0 + Base::koff();
    if (VEC) {
      int rr = 0, s = 0, c = 0;
      const bool kin = kk < kend;
      if (kin) {
        const int sc = S * C;
        rr = (int)(kk / sc);
        const int rem = (int)(kk - (int64_t)rr * sc);
        s = rem / C;
        c = rem - s * C;
      }
#pragma unroll
      for (int j = 0; j < Base::kN; ++j) {
        const int h = h_[j] + rr, w = w_[j] + s;
        const bool ok = kin && n_[j] >= 0 && h >= 0 && h < H && w >= 0 && w < W;
        r[j] = ok ? *reinterpret_cast<const float4*>(
                        &x[(((int64_t)n_[j] * H + h) * W + w) * C + c])
                  : zero4();
      }
    } else {
#pragma unroll
      for (int j = 0; j < Base::kN; ++j) {
        r[j].x = at(j, kk + 0, kend);
        r[j].y = at(j, kk + 1, kend);
        r[j].z = at(j, kk + 2, kend);
        r[j].w = at(j, kk + 3, kend);
      }
    }
  }
};

// Convolution input gradient, A = output gradient through the taps:
// A[m = (n, h, w)][kk = (r, s, k)] = dY[n][p][q][k] with p st = h + pad - r,
// q st = w + pad - s (zero when not an exact, in-range output position).
// Row-of-k; VEC needs K % 4 == 0.
template <int E, bool VEC>
struct ConvGradTap : RowK<E> {
  using Base = RowK<E>;
  const float* dy;
  int H, W, K, S, st, pad, P, Q;
  int64_t M;
  int n_[Base::kN], h_[Base::kN], w_[Base::kN];   // per row: image, h + pad, w + pad
  __device__ void init(int64_t mn0, int64_t MN) {
    M = MN;
#pragma unroll
    for (int j = 0; j < Base::kN; ++j) {
      const int64_t m = mn0 + Base::row(j);
      if (m < M) {
        const int64_t hw = (int64_t)H * W;
        const int n = (int)(m / hw);
        const int rem = (int)(m - (int64_t)n * hw);
        const int h = rem / W, w = rem - h * W;
        n_[j] = n;
        h_[j] = h + pad;
        w_[j] = w + pad;
      } else {
        n_[j] = -1;
      }
    }
  }
  __device__ float at(int j, int64_t kk, int64_t kend) const {
    if (n_[j] < 0 || kk >= kend) return 0.f;
    const int sk = S * K;
    const int r = (int)(kk / sk);
    const int rem = (int)(kk - (int64_t)r * sk);
    const int s = rem / K, k = rem - s * K;
    const int ph = h_[j] - r, qw = w_[j] - s;
    if (ph < 0 || qw < 0 || ph % st || qw % st) return 0.f;
    const int p = ph / st, q = qw / st;
    if (p >= P || q >= Q) return 0.f;
    return dy[(((int64_t)n_[j] * P + p) * Q + q) * K + k];
  }
  __device__ void fetch(int64_t k0, int64_t kend, float4 (&r)[Base::kN]) const {
    const int64_t kk = k0 + Base::koff();
    if (VEC) {
      int rr = 0, s = 0, k = 0;
      const bool kin = kk < kend;
      if (kin) {
        const int sk = S * K;
        rr = (int)(kk / sk);
        const int rem = (int)(kk - (int64_t)rr * sk);
        s = rem / K;
        k = rem - s * K;
      }
#pragma unroll
      for (int j = 0; j < Base::kN; ++j) {
        const int ph = h_[j] - rr, qw = w_[j] - s;
        bool ok = kin && n_[j] >= 0 && ph >= 0 && qw >= 0 && ph % st == 0 && qw % st == 0;
        const int p = ok ? ph / st : 0, q = ok ? qw / st : 0;
        ok = ok && p < P && q < Q;
        r[j] = ok ? *reinterpret_cast<const float4*>(
                        &dy[(((int64_t)n_[j] * P + p) * Q + q) * K + k])
                  : zero4();
      }
    } else {
#pragma unroll
      for (int j = 0; j < Base::kN; ++j) {
        r[j].x = at(j, kk + 0, kend);
        r[j].y = at(j, kk + 1, kend);
        r[j].z = at(j, kk + 2, kend);
        r[j].w = at(j, kk + 3, kend);
      }
    }
  }
};

// Convolution input gradient, B = filter seen per tap:
// B[kk = (r, s, k)][c] = W[k][r][s][c]   (row-of-m; needs C % 4 == 0)
template <int E>
struct ConvFilterTap : RowM<E> {
  using Base = RowM<E>;
  const float* w;
  int C, K, R, S;
  int64_t c0;
  __device__ void init(int64_t mn0, int64_t) { c0 = mn0 + Base::moff(); }
  __device__ void fetch(int64_t k0, int64_t kend, float4 (&r)[Base::kN]) const {
#pragma unroll
    for (int j = 0; j < Base::kN; ++j) {
      const int64_t kk = k0 + Base::krow(j);
      if (kk < kend && c0 < C) {
        const int sk = S * K;
        const int rr = (int)(kk / sk);
        const int rem = (int)(kk - (int64_t)rr * sk);
        const int s = rem / K, k = rem - s * K;
        r[j] = *reinterpret_cast<const float4*>(&w[(((int64_t)k * R + rr) * S + s) * C + c0]);
      } else {
        r[j] = zero4();
      }
    }
  }
};

// Convolution filter gradient, B = input patches along the pixel axis:
// B[kk = (n, p, q)][col = (r, s, c)] = X[n][p st - pad + r][q st - pad + s][c]
// (row-of-m; VEC needs C % 4 == 0)
template <int E, bool VEC>
struct ConvPixelPatch : RowM<E> {
  using Base = RowM<E>;
  const float* x;
  int H, W, C, S, st, pad, P, Q;
  int64_t RSC;
  int r_[4], s_[4], c_[4];   // per column of this thread; r = -1: no column
  __device__ void init(int64_t mn0, int64_t MN) {
    RSC = MN;
    const int64_t col = mn0 + Base::moff();
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int64_t cc = col + e;
      if (cc < RSC && (VEC ? e == 0 : true)) {
        const int sc = S * C;
        const int r = (int)(cc / sc);
        const int rem = (int)(cc - (int64_t)r * sc);
        r_[e] = r;
        s_[e] = rem / C;
        c_[e] = rem - s_[e] * C;
      } else {
        r_[e] = -1;
      }
    }
  }
  __device__ void fetch(int64_t k0, int64_t kend, float4 (&r)[Base::kN]) const {
#pragma unroll
    for (int j = 0; j < Base::kN; ++j) {
      const int64_t kk = k0 + Base::krow(j);
      r[j] = zero4();
      if (kk >= kend) continue;
      const int64_t pq = (int64_t)P * Q;
      const int n = (int)(kk / pq);
      const int rem = (int)(kk - (int64_t)n * pq);
      const int p = rem / Q, q = rem - p * Q;
      const int hb = p * st - pad, wb = q * st - pad;
      if (VEC) {
        const int h = hb + r_[0], w = wb + s_[0];
        if (r_[0] >= 0 && h >= 0 && h < H && w >= 0 && w < W)
          r[j] = *reinterpret_cast<const float4*>(&x[(((int64_t)n * H + h) * W + w) * C + c_[0]]);
      } else {
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int h = hb + r_[e], w = wb + s_[e];
          v[e] = (r_[e] >= 0 && h >= 0 && h < H && w >= 0 && w < W)
                     ? x[(((int64_t)n * H + h) * W + w) * C + c_[e]]
                     : 0.f;
        }
        r[j] = make_float4(v[0], v[1], v[2], v[3]);
      }
    }
  }
};

// ---------------------------------------------------------------- kernel
template <class L>
__device__ inline float4 read_op(const float* lds, int i, int k) {
  if (L::kRowOfK) return *reinterpret_cast<const float4*>(&lds[i * LDK + k]);
  constexpr int ld = L::kRowOfK ? LDK : (L::kLds / BK);
  return make_float4(lds[(k + 0) * ld + i], lds[(k + 1) * ld + i], lds[(k + 2) * ld + i],
                     lds[(k + 3) * ld + i]);
}

__device__ inline float comp(const float4& v, int t) {
  return t == 0 ? v.x : t == 1 ? v.y : t == 2 ? v.z : v.w;
}

// BM x BN tile; the four waves form a 2 x 2 grid of (BM/2) x (BN/2) sub-tiles,
// each made of (BM/64) x (BN/64) MFMA 32 x 32 blocks.
// Batched problems (grid z): batch z = (zo, zi) with zi = z mod inner; operand
// and result pointers move by zo * outer stride + zi * inner stride.
struct Batch {
  int64_t inner;
  int64_t a_o, a_i, b_o, b_i, c_o, c_i;
};

template <class L>
__device__ inline void shift(L& l, int64_t d) {
  l.p += d;
}

// rowsum (optional): rowsum[slice][m] = sum over this slice's k of A[m][k]
template <int BM, int BN, class LA, class LB, bool BIAS, bool BATCHED>
__global__ __launch_bounds__(THREADS) void gemm_kernel(LA la, LB lb, float* __restrict__ c,
                                                       int64_t ldc, int64_t slice_stride,
                                                       const float* __restrict__ bias, int64_t M,
                                                       int64_t N, int64_t K, int64_t k_slice,
                                                       int tiles_m, int tiles_n, Batch bt,
                                                       float* __restrict__ rowsum) {
  constexpr int MB = BM / 64, NB = BN / 64;
  if constexpr (BATCHED) {
    const int64_t z = blockIdx.z, zo = z / bt.inner, zi = z % bt.inner;
    shift(la, zo * bt.a_o + zi * bt.a_i);
    shift(lb, zo * bt.b_o + zi * bt.b_i);
    c += zo * bt.c_o + zi * bt.c_i;
  }
  __shared__ __attribute__((aligned(16))) float As[2][LA::kLds];
  __shared__ __attribute__((aligned(16))) float Bs[2][LB::kLds];

  // grouped tile order: 8 tile-rows share their B tiles in L2
  const int t = blockIdx.x;
  const int group = 8;
  const int per_group = group * tiles_n;
  const int g = t / per_group;
  const int first_m = g * group;
  const int gsize = min(tiles_m - first_m, group);
  const int tm = first_m + (t % per_group) % gsize;
  const int tn = (t % per_group) / gsize;
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const int64_t kb = (int64_t)blockIdx.y * k_slice;
  const int64_t ke = min(K, kb + k_slice);

  la.init(m0, M);
  lb.init(n0, N);
  float4 ra[LA::kN], rb[LB::kN];
  floatx16 acc[MB][NB];
#pragma unroll
  for (int a = 0; a < MB; ++a)
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  const bool sums = rowsum != nullptr && tn == 0 && (int)threadIdx.x < BM;
  float rs = 0.f;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int half = lane >> 5;
  const int li = lane & 31;

  if (kb < ke) {
    la.fetch(kb, ke, ra);
    lb.fetch(kb, ke, rb);
    LA::store(As[0], ra);
    LB::store(Bs[0], rb);
  }
  __syncthreads();
  int buf = 0;
  for (int64_t k0 = kb; k0 < ke; k0 += BK) {
    const bool more = k0 + BK < ke;
    if (more) {
      la.fetch(k0 + BK, ke, ra);
      lb.fetch(k0 + BK, ke, rb);
    }
    const float* A = As[buf];
    const float* B = Bs[buf];
    if (sums) {
#pragma unroll
      for (int k = 0; k < BK; ++k) {
        if constexpr (LA::kRowOfK) rs += A[threadIdx.x * LDK + k];
        else rs += A[k * (LA::kLds / BK) + threadIdx.x];
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int kq = half * 16 + 4 * j;
      float4 a[MB], b[NB];
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) a[mb] = read_op<LA>(A, wm * (BM / 2) + mb * 32 + li, kq);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) b[nb] = read_op<LB>(B, wn * (BN / 2) + nb * 32 + li, kq);
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(comp(a[mb], s), comp(b[nb], s),
                                                              acc[mb][nb], 0, 0, 0);
    }
    if (more) {
      LA::store(As[buf ^ 1], ra);
      LB::store(Bs[buf ^ 1], rb);
    }
    __syncthreads();
    buf ^= 1;
  }

  if (sums && m0 + threadIdx.x < M) rowsum[(int64_t)blockIdx.y * M + m0 + threadIdx.x] = rs;
  float* out = c + (int64_t)blockIdx.y * slice_stride;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int64_t col = n0 + wn * (BN / 2) + nb * 32 + li;
      if (col >= N) continue;
      const float bv = BIAS ? bias[col] : 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + wm * (BM / 2) + mb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (row < M) out[row * ldc + col] = acc[mb][nb][r] + bv;
      }
    }
}

template <int BM, int BN, class LA, class LB, bool BIAS, bool BATCHED = false>
hipError_t run_gemm(const LA& la, const LB& lb, float* c, int64_t ldc, const float* bias,
                    int64_t M, int64_t N, int64_t K, int64_t slices, hipStream_t s,
                    int64_t batches = 1, Batch bt = Batch{1, 0, 0, 0, 0, 0, 0},
                    float* rowsum = nullptr) {
  const int64_t tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  if (tiles_m * tiles_n > INT32_MAX / 2 || slices > 65535 || batches > 65535 || batches < 1)
    return hipErrorInvalidValue;
  int64_t k_slice = (K + slices - 1) / slices;
  k_slice = (k_slice + BK - 1) / BK * BK;
  dim3 grid((unsigned)(tiles_m * tiles_n), (unsigned)slices, (unsigned)batches);
  hipLaunchKernelGGL((gemm_kernel<BM, BN, LA, LB, BIAS, BATCHED>), grid, dim3(THREADS), 0, s, la,
                     lb, c, ldc, M * ldc, bias, M, N, K, k_slice, (int)tiles_m, (int)tiles_n, bt,
                     rowsum);
  return hipGetLastError();
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// Tile shape: 128 x 128, or 64 along a dimension that is at most 64 wide
// (half of a 128-wide tile would compute zeros).
enum Shape { S128x128, S128x64, S64x128 };
Shape pick_shape(int64_t M, int64_t N) {
  if (N <= 64 && M > 64) return S128x64;
  if (M <= 64) return S64x128;
  return S128x128;
}

// Runs the GEMM with loader templates A<E>, B<E> instantiated for the chosen
// tile shape; `make_a(tag)` / `make_b(tag)` build them.
template <template <int> class LAT, template <int> class LBT, bool BIAS, bool BATCHED = false,
          class FA, class FB>
hipError_t dispatch(FA fa, FB fb, float* c, int64_t ldc, const float* bias, int64_t M, int64_t N,
                    int64_t K, int64_t slices, hipStream_t s, int64_t batches = 1,
                    Batch bt = Batch{1, 0, 0, 0, 0, 0, 0}, float* rowsum = nullptr) {
  switch (pick_shape(M, N)) {
    case S128x64: {
      LAT<128> a{};
      LBT<64> b{};
      fa(a);
      fb(b);
      return run_gemm<128, 64, LAT<128>, LBT<64>, BIAS, BATCHED>(a, b, c, ldc, bias, M, N, K,
                                                                 slices, s, batches, bt, rowsum);
    }
    case S64x128: {
      LAT<64> a{};
      LBT<128> b{};
      fa(a);
      fb(b);
      return run_gemm<64, 128, LAT<64>, LBT<128>, BIAS, BATCHED>(a, b, c, ldc, bias, M, N, K,
                                                                 slices, s, batches, bt, rowsum);
    }
    default: {
      LAT<128> a{};
      LBT<128> b{};
      fa(a);
      fb(b);
      return run_gemm<128, 128, LAT<128>, LBT<128>, BIAS, BATCHED>(a, b, c, ldc, bias, M, N, K,
                                                                   slices, s, batches, bt, rowsum);
    }
  }
}

template <int E> using MatKv = MatK<E, true>;
template <int E> using MatKs = MatK<E, false>;
template <int E> using MatMv = MatM<E, true>;
template <int E> using MatMs = MatM<E, false>;
template <int E> using ConvPatchV = ConvPatch<E, true>;
template <int E> using ConvPatchS = ConvPatch<E, false>;
template <int E> using ConvGradTapV = ConvGradTap<E, true>;
template <int E> using ConvGradTapS = ConvGradTap<E, false>;
template <int E> using ConvPixelPatchV = ConvPixelPatch<E, true>;
template <int E> using ConvPixelPatchS = ConvPixelPatch<E, false>;

// ---------------------------------------------------------------- small kernels
// out[j] = sum over slices of part[s][j]: four interleaved accumulators
// (slices s = u mod 4), added in a fixed order
__global__ void slice_sum_kernel(const float* __restrict__ part, float* __restrict__ out,
                                 int64_t n, int64_t slices) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= n) return;
  float a[4] = {0.f, 0.f, 0.f, 0.f};
  int64_t s = 0;
  for (; s + 4 <= slices; s += 4) {
#pragma unroll
    for (int u = 0; u < 4; ++u) a[u] += part[(s + u) * n + j];
  }
  for (; s < slices; ++s) a[0] += part[s * n + j];
  out[j] = (a[0] + a[1]) + (a[2] + a[3]);
}

}  // namespace

// ---------------------------------------------------------------- launchers
hipError_t linear_fwd(const float* X, const float* W, const float* b, float* Y, int64_t M,
                      int64_t K, int64_t N, hipStream_t s) {
  auto fa = [&](auto& a) { a.p = X; a.ld = K; };
  auto fb = [&](auto& bb) { bb.p = W; bb.ld = K; };
  if (K % 4 == 0 && aligned16(X) && aligned16(W))
    return dispatch<MatKv, MatKv, true>(fa, fb, Y, N, b, M, N, K, 1, s);
  return dispatch<MatKs, MatKs, true>(fa, fb, Y, N, b, M, N, K, 1, s);
}

hipError_t linear_bwd_x(const float* W, const float* dY, float* dX, int64_t M, int64_t K,
                        int64_t N, hipStream_t s) {
  // dX[M][K] = dY[M][N] W[N][K]: A = dY (contiguous along the reduction), B[n_out][k_in] = W
  auto fa = [&](auto& a) { a.p = dY; a.ld = N; };
  auto fb = [&](auto& bb) { bb.p = W; bb.ld = K; };
  if (N % 4 == 0 && K % 4 == 0 && aligned16(W) && aligned16(dY))
    return dispatch<MatKv, MatMv, false>(fa, fb, dX, K, nullptr, M, K, N, 1, s);
  return dispatch<MatKs, MatMs, false>(fa, fb, dX, K, nullptr, M, K, N, 1, s);
}

hipError_t linear_bwd_w(const float* X, const float* dY, float* dW, float* db, float* part,
                        int64_t slices, int64_t M, int64_t K, int64_t N, hipStream_t s) {
  // dW[N][K] = dY^T X: A[n][m] = dY[m][n] (contiguous in n), B[m][k] = X[m][k] (contiguous in k);
  // db = the row sums of A.  With slices > 1, part holds slices copies of dW, then slices of db.
  if (slices > 1 && part == nullptr) return hipErrorInvalidValue;
  float* out = slices > 1 ? part : dW;
  float* sums = slices > 1 ? part + slices * N * K : db;
  auto fa = [&](auto& a) { a.p = dY; a.ld = N; };
  auto fb = [&](auto& bb) { bb.p = X; bb.ld = K; };
  const Batch one{1, 0, 0, 0, 0, 0, 0};
  hipError_t e;
  if (N % 4 == 0 && K % 4 == 0 && aligned16(X) && aligned16(dY))
    e = dispatch<MatMv, MatMv, false>(fa, fb, out, K, nullptr, N, K, M, slices, s, 1, one, sums);
  else
    e = dispatch<MatMs, MatMs, false>(fa, fb, out, K, nullptr, N, K, M, slices, s, 1, one, sums);
  if (e != hipSuccess || slices <= 1) return e;
  hipLaunchKernelGGL(slice_sum_kernel, dim3((unsigned)((N * K + 255) / 256)), dim3(256), 0, s,
                     part, dW, N * K, slices);
  hipLaunchKernelGGL(slice_sum_kernel, dim3((unsigned)((N + 255) / 256)), dim3(256), 0, s, sums, db,
                     N, slices);
  return hipGetLastError();
}

hipError_t gemm_batched(bool a_rowk, const float* A, int64_t lda, bool b_rowk, const float* B,
                        int64_t ldb, float* C, int64_t ldc, int64_t M, int64_t N, int64_t K,
                        int64_t batches, const BatchStrides& st, hipStream_t s) {
  const Batch bt{st.inner, st.a_outer, st.a_inner, st.b_outer, st.b_inner, st.c_outer,
                 st.c_inner};
  auto fa = [&](auto& a) { a.p = A; a.ld = lda; };
  auto fb = [&](auto& b) { b.p = B; b.ld = ldb; };
  const bool vec = lda % 4 == 0 && ldb % 4 == 0 && aligned16(A) && aligned16(B) &&
                   (a_rowk ? K % 4 == 0 : M % 4 == 0) && (b_rowk ? K % 4 == 0 : N % 4 == 0) &&
                   st.a_outer % 4 == 0 && st.a_inner % 4 == 0 && st.b_outer % 4 == 0 &&
                   st.b_inner % 4 == 0;
#define GEMM_BATCHED_CASE(LA, LB) \
  return dispatch<LA, LB, false, true>(fa, fb, C, ldc, nullptr, M, N, K, 1, s, batches, bt)
  if (vec) {
    if (a_rowk && b_rowk) GEMM_BATCHED_CASE(MatKv, MatKv);
    if (a_rowk) GEMM_BATCHED_CASE(MatKv, MatMv);
    if (b_rowk) GEMM_BATCHED_CASE(MatMv, MatKv);
    GEMM_BATCHED_CASE(MatMv, MatMv);
  }
  if (a_rowk && b_rowk) GEMM_BATCHED_CASE(MatKs, MatKs);
  if (a_rowk) GEMM_BATCHED_CASE(MatKs, MatMs);
  if (b_rowk) GEMM_BATCHED_CASE(MatMs, MatKs);
  GEMM_BATCHED_CASE(MatMs, MatMs);
#undef GEMM_BATCHED_CASE
}

hipError_t conv_fwd(const float* X, const float* W, float* Y, const ConvShape& c, hipStream_t s) {
  const int64_t M = c.N * c.P * c.Q, N = c.K, K = c.R * c.S * c.C;
  auto fa = [&](auto& a) {
    a.x = X; a.H = (int)c.H; a.W = (int)c.W; a.C = (int)c.C; a.S = (int)c.S;
    a.st = (int)c.stride; a.pad = (int)c.pad; a.P = (int)c.P; a.Q = (int)c.Q;
  };
  auto fb = [&](auto& b) { b.p = W; b.ld = K; };
  if (c.C % 4 == 0) return dispatch<ConvPatchV, MatKv, false>(fa, fb, Y, N, nullptr, M, N, K, 1, s);
  return dispatch<ConvPatchS, MatKs, false>(fa, fb, Y, N, nullptr, M, N, K, 1, s);
}

hipError_t conv_bwd_x(const float* W, const float* dY, float* dX, const ConvShape& c,
                      hipStream_t s) {
  if (c.C % 4 != 0) return hipErrorInvalidValue;   // every conv with an input gradient has C % 4 == 0
  const int64_t M = c.N * c.H * c.W, N = c.C, K = c.R * c.S * c.K;
  auto fa = [&](auto& a) {
    a.dy = dY; a.H = (int)c.H; a.W = (int)c.W; a.K = (int)c.K; a.S = (int)c.S;
    a.st = (int)c.stride; a.pad = (int)c.pad; a.P = (int)c.P; a.Q = (int)c.Q;
  };
  auto fb = [&](auto& b) {
    b.w = W; b.C = (int)c.C; b.K = (int)c.K; b.R = (int)c.R; b.S = (int)c.S;
  };
  if (c.K % 4 == 0)
    return dispatch<ConvGradTapV, ConvFilterTap, false>(fa, fb, dX, N, nullptr, M, N, K, 1, s);
  return dispatch<ConvGradTapS, ConvFilterTap, false>(fa, fb, dX, N, nullptr, M, N, K, 1, s);
}

hipError_t conv_bwd_w(const float* X, const float* dY, float* dW, float* part, int64_t slices,
                      const ConvShape& c, hipStream_t s) {
  // dW[K][RSC] = sum over pixels of dY[pixel][k] * patch[pixel][rsc]
  const int64_t M = c.K, N = c.R * c.S * c.C, K = c.N * c.P * c.Q;
  float* out = slices > 1 ? part : dW;
  auto fa = [&](auto& a) { a.p = dY; a.ld = c.K; };
  auto fb = [&](auto& b) {
    b.x = X; b.H = (int)c.H; b.W = (int)c.W; b.C = (int)c.C; b.S = (int)c.S;
    b.st = (int)c.stride; b.pad = (int)c.pad; b.P = (int)c.P; b.Q = (int)c.Q;
  };
  hipError_t e;
  if (c.K % 4 == 0) {
    if (c.C % 4 == 0)
      e = dispatch<MatMv, ConvPixelPatchV, false>(fa, fb, out, N, nullptr, M, N, K, slices, s);
    else
      e = dispatch<MatMv, ConvPixelPatchS, false>(fa, fb, out, N, nullptr, M, N, K, slices, s);
  } else {
    e = dispatch<MatMs, ConvPixelPatchS, false>(fa, fb, out, N, nullptr, M, N, K, slices, s);
  }
  if (e != hipSuccess || slices <= 1) return e;
  const int64_t n = M * N;
  hipLaunchKernelGGL(slice_sum_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, part,
                     dW, n, slices);
  return hipGetLastError();
}

}  // namespace ooc
