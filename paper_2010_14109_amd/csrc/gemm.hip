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
// padding.  Loaders keep per-row offsets from their set-up, so a K tile costs
// one add per row; a convolution whose channel count is a multiple of 32 has
// every K tile inside one filter tap (uniform over the workgroup), and the
// remaining index splits use multiply-high division by invariant integers.
// The input gradient of a strided convolution is computed per stride class
// of input pixels (h mod st, w mod st), each class a GEMM over only the taps
// that reach it.  LDS layout follows the contiguous direction: "row of k" tiles
// ([rows][32], k quads XOR-swizzled by row against bank conflicts) are
// written and read with 16-byte accesses, "row of m" tiles ([32][rows]) are
// written with 16-byte accesses and read with 4-byte ones.  No padding: the
// 128 x 64 tiles then fit three workgroups in a CU's 160 KB of LDS.
//
// Split-K: the filter gradients reduce over N P Q pixels or over the rows of
// a dense layer (up to millions), so the grid's second dimension cuts that
// axis into slices whose partial tiles go to separate buffers and are summed
// afterwards in slice order.  A dense layer's bias gradient (the column sums
// of dY) is taken from the A tiles already in LDS by the workgroups of the
// first tile column, slice by slice like dW.  No atomics anywhere: results
// do not depend on scheduling or addresses.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <type_traits>

#include "kernels.h"

namespace ooc {

namespace {

constexpr int BK = 32;
constexpr int THREADS = 256;
constexpr uint32_t kXcds = 8;   // accelerator complex dies of an MI355X, one L2 each

typedef float floatx16 __attribute__((ext_vector_type(16)));

__device__ inline float4 zero4() { return make_float4(0.f, 0.f, 0.f, 0.f); }

// ---------------------------------------------------------------- loaders
// A loader feeds one operand tile of extent E (tile rows along m or n) by 32
// along k.  init(mn0, MN) runs once per workgroup (mn0 = tile origin, MN =
// extent of the matrix), fetch(k0, kend, r) loads this thread's E / 8 values
// of the K tile starting at k0 as E / 32 float4, store(lds, r) writes them.
//
// No load sits behind a branch, so that the address arithmetic of the next
// tile can be scheduled between the MFMAs of the current one.  Values at
// k >= kend must be zero (they enter every dot product): their lanes load
// from a block of zeros instead.  Rows and columns past M or N only reach C
// entries that are never stored, so their lanes read a clamped in-range
// address and whatever they load is harmless.  Zero padding of a
// convolution is masked like k >= kend.
//
// Row-of-k layout [E][32] (swizzled, below): thread t loads rows (t >> 3) + 32 j,
// k offset (t & 7) * 4.  Row-of-m layout [32][E], two thread maps: RowM has E / 4
// threads per k row, thread t loading k rows t / (E / 4) + (1024 / E) j at m
// offset (t % (E / 4)) * 4, so that a wave reads whole rows; RowM1 gives
// thread t the single k row t >> 3 and its E / 8 consecutive m values from
// (t & 7) E / 8 on, so that one row address serves all of its loads (for
// views whose row addresses are costly to form).

// What masked lanes load (never written).
__device__ __attribute__((aligned(16))) float g_zero[64] = {};

__device__ inline float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }

// Pins v in a register at this point.  The compiler would otherwise move an
// address computation that only a masked select uses into a branch around
// it, which is what the loaders avoid.
template <class T>
__device__ inline void keep(T& v) {
  asm volatile("" : "+v"(v));
}

// Row-of-k tiles [E][32] keep k quad q of row i in slot q ^ (i mod 8): the
// lanes of a 16-byte read take 8 consecutive rows at one quad, which then
// cover all banks, without padding the rows.
__device__ inline int rowk_index(int i, int k) { return i * BK + ((((k >> 2) ^ i) & 7) << 2) + (k & 3); }

template <int E>
struct RowK {
  static constexpr bool kRowOfK = true;
  static constexpr int kN = E / 32;
  static constexpr int kLds = E * BK;
  __device__ static int row(int j) { return (threadIdx.x >> 3) + 32 * j; }
  __device__ static int koff() { return (threadIdx.x & 7) * 4; }
  __device__ static void store(float* lds, const float4 (&r)[kN]) {
#pragma unroll
    for (int j = 0; j < kN; ++j)
      *reinterpret_cast<float4*>(&lds[rowk_index(row(j), koff())]) = r[j];
  }
};
template <int E>
struct RowM {
  static constexpr bool kRowOfK = false;
  static constexpr int kN = E / 32;
  static constexpr int kLd = E;
  static constexpr int kLds = BK * kLd;
  __device__ static int krow(int j) { return (int)threadIdx.x / (E / 4) + (1024 / E) * j; }
  __device__ static int moff() { return ((int)threadIdx.x % (E / 4)) * 4; }
  __device__ static void store(float* lds, const float4 (&r)[kN]) {
#pragma unroll
    for (int j = 0; j < kN; ++j) *reinterpret_cast<float4*>(&lds[krow(j) * kLd + moff()]) = r[j];
  }
};
template <int E>
struct RowM1 {
  static constexpr bool kRowOfK = false;
  static constexpr int kN = E / 32;
  static constexpr int kLd = E;
  static constexpr int kLds = BK * kLd;
  __device__ static int krow() { return (int)threadIdx.x >> 3; }
  __device__ static int moff() { return ((int)threadIdx.x & 7) * (E / 8); }
  __device__ static void store(float* lds, const float4 (&r)[kN]) {
#pragma unroll
    for (int j = 0; j < kN; ++j)
      *reinterpret_cast<float4*>(&lds[krow() * kLd + moff() + 4 * j]) = r[j];
  }
};

// x / d for 0 <= x < 2^31 and an invariant d >= 1 with one multiply-high
// (Granlund and Montgomery, division by invariant integers using
// multiplication, 1994): with l = ceil(log2 d) and m = floor(2^(31+l) / d) + 1,
// 2^(31+l) < m d <= 2^(31+l) + 2^l, hence floor(x m / 2^(31+l)) = floor(x / d)
// for every x < 2^31, and m < 2^32.  d = 1 takes m = 2^32 - 1 and adds one
// to x first: floor((x + 1)(2^32 - 1) / 2^32) = x for x + 1 <= 2^32.  Both
// cases are the same instructions, so a division never branches.
struct FastDiv {
  uint32_t d = 1, m = 0xffffffffu, s = 0, a = 1;
  static FastDiv make(int64_t dv) {
    FastDiv f;
    f.d = (uint32_t)dv;
    if (dv <= 1) return f;
    uint32_t l = 0;
    while ((1ull << l) < (uint64_t)dv) ++l;
    f.m = (uint32_t)((1ull << (31 + l)) / (uint64_t)dv + 1);
    f.s = l - 1;
    f.a = 0;
    return f;
  }
  __device__ int div(int x) const { return (int)(__umulhi((uint32_t)x + a, m) >> s); }
};

constexpr int kFar = -(1 << 29);   // coordinate of a row past the matrix: fails every bounds check

__device__ inline bool inside(int v, int n) { return (unsigned)v < (unsigned)n; }

// X[i][k] = p[i * ld + k]  (contiguous along k)
template <int E, bool VEC>
struct MatK : RowK<E> {
  using Base = RowK<E>;
  const float* p;
  int64_t ld;
  int64_t off_[Base::kN];   // (row, clamped to the matrix) * ld + this lane's k offset
  __device__ void init(int64_t mn0, int64_t MN) {
#pragma unroll
    for (int j = 0; j < Base::kN; ++j) {
      const int64_t i = mn0 + Base::row(j);
      off_[j] = (i < MN ? i : 0) * ld + Base::koff();
    }
  }
  __device__ void fetch(int64_t k0, int64_t kend, float4 (&r)[Base::kN]) const {
    const int64_t k = k0 + Base::koff();
#pragma unroll
    for (int j = 0; j < Base::kN; ++j) {
      const float* q = p + off_[j] + k0;
      if (VEC) {
        r[j] = ld4(k < kend ? q : g_zero);
      } else {
        r[j].x = *(k + 0 < kend ? q + 0 : g_zero);
        r[j].y = *(k + 1 < kend ? q + 1 : g_zero);
        r[j].z = *(k + 2 < kend ? q + 2 : g_zero);
        r[j].w = *(k + 3 < kend ? q + 3 : g_zero);
      }
    }
  }
};

// X[i][k] = p[k * ld + i]  (contiguous along m or n; VEC needs MN % 4 == 0)
template <int E, bool VEC>
struct MatM : RowM<E> {
  using Base = RowM<E>;
  const float* p;
  int64_t ld;
  int64_t i0;                // this lane's first m
  int64_t rows;              // MN
  int64_t off_[Base::kN];    // k row * ld (+ the m offset clamped to the matrix, VEC)
  __device__ void init(int64_t mn0, int64_t MN) {
    i0 = mn0 + Base::moff();
    rows = MN;
#pragma unroll
    for (int j = 0; j < Base::kN; ++j)
      off_[j] = Base::krow(j) * ld + (VEC ? (i0 < MN ? i0 : 0) : 0);
  }
  __device__ void fetch(int64_t k0, int64_t kend, float4 (&r)[Base::kN]) const {
    const float* pk = p + k0 * ld;
#pragma unroll
    for (int j = 0; j < Base::kN; ++j) {
      const bool ok = k0 + Base::krow(j) < kend;
      if (VEC) {
        r[j] = ld4(ok ? pk + off_[j] : g_zero);
      } else {
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int64_t i = i0 + e;
          v[e] = *(ok ? pk + off_[j] + (i < rows ? i : 0) : g_zero);
        }
        r[j] = make_float4(v[0], v[1], v[2], v[3]);
      }
    }
  }
};

// Loader modes of the convolution views.  Row-of-k views: TAP when the
// reduced channel count is a multiple of 32 (a K tile lies inside one filter
// tap, uniform over the workgroup), VEC4 when it is a multiple of 4 (each lane
// splits its own k index, four consecutive channels per load), SCALAR
// otherwise.  Row-of-m views: TAP when all E / 8 values of a lane lie in one
// tap (channels a multiple of 16), VEC4 when each float4 does.
enum { SCALAR = 0, VEC4 = 1, TAP = 2 };

// Convolution forward, A = input patches: A[m = (n, p, q)][kk = (r, s, c)] =
// X[n][p st - pad + r][q st - pad + s][c]   (row-of-k)
template <int E, int MODE>
struct ConvPatch : RowK<E> {
  using Base = RowK<E>;
  const float* x;
  int H, W, C, S, st, pad;
  FastDiv dQ, dPQ, dC, dS, dSC;   // by Q, P Q, C, S, S C
  int64_t base_[Base::kN];        // offset of X[n][h0][w0][0]
  int h_[Base::kN], w_[Base::kN]; // h0 = p st - pad, w0 = q st - pad
  __device__ void init(int64_t mn0, int64_t M) {
#pragma unroll
    for (int j = 0; j < Base::kN; ++j) {
      const int64_t m = mn0 + Base::row(j);
      if (m < M) {
        const int n = dPQ.div((int)m);
        const int rem = (int)m - n * (int)dPQ.d;
        const int p = dQ.div(rem), q = rem - p * (int)dQ.d;
        h_[j] = p * st - pad;
        w_[j] = q * st - pad;
        base_[j] = (((int64_t)n * H + h_[j]) * W + w_[j]) * C;
      } else {
        h_[j] = kFar;
        w_[j] = 0;
        base_[j] = 0;
      }
    }
  }
  // value at (row j, column kk) or 0 when kk >= kend or outside the image
  __device__ float at(int j, int kk, int64_t kend) const {
    const bool kin = kk < kend;
    const int kc = kin ? kk : 0;
    const int r = dSC.div(kc);
    const int rem = kc - r * (int)dSC.d;
    const int s = dC.div(rem), c = rem - s * C;
    const bool ok = kin & inside(h_[j] + r, H) & inside(w_[j] + s, W);
    return *(ok ? x + base_[j] + ((int64_t)r * W + s) * C + c : g_zero);
  }
  __device__ void fetch(int64_t k0, int64_t kend, float4 (&r)[Base::kN]) const {
    const int kk = (int)k0 + Base::koff();
    if constexpr (MODE == SCALAR) {
#pragma unroll
      for (int j = 0; j < Base::kN; ++j)
        r[j] = make_float4(at(j, kk, kend), at(j, kk + 1, kend), at(j, kk + 2, kend),
                           at(j, kk + 3, kend));
    } else {
      int rr, s, c;
      if constexpr (MODE == TAP) {   // uniform tap
        const int tap = dC.div((int)k0);
        rr = dS.div(tap);
        s = tap - rr * S;
        c = (int)k0 - tap * C + Base::koff();
      } else {
        rr = dSC.div(kk);
        const int rem = kk - rr * (int)dSC.d;
        s = dC.div(rem);
        c = rem - s * C;
      }
      const int64_t toff = ((int64_t)rr * W + s) * C + c;
      const bool kin = kk < kend;
#pragma unroll
      for (int j = 0; j < Base::kN; ++j) {
        const bool ok = kin & inside(h_[j] + rr, H) & inside(w_[j] + s, W);
        r[j] = ld4(ok ? x + base_[j] + toff : g_zero);
      }
    }
  }
};

// Convolution input gradient for the input pixels of one stride class,
// h = st hh + ph and w = st ww + pw (hh < Hc, ww < Wc).  Only the taps
// r = r0 + st i (i < nR) and s = s0 + st j (j < nS) reach them, from the
// output position p = hh + a - i, q = ww + b - j (a = (ph + pad - r0) / st,
// b = (pw + pad - s0) / st); A is the output gradient gathered that way:
// A[m = (n, hh, ww)][kk = (i, j, k)] = dY[n][hh + a - i][ww + b - j][k], zero
// outside the output.  Stride 1 is the single class r0 = s0 = 0, a = b = pad.
// Row-of-k; the mode refers to the output channels K.
template <int E, int MODE>
struct ConvGradTap : RowK<E> {
  using Base = RowK<E>;
  const float* dy;
  int P, Q, K, nS, a, b;
  FastDiv dWc, dHWc, dK, dnS, dSK;   // by Wc, Hc Wc, K, nS, nS K
  int64_t base_[Base::kN];           // offset of dY[n][hh + a][ww + b][0]
  int p_[Base::kN], q_[Base::kN];    // hh + a, ww + b
  __device__ void init(int64_t mn0, int64_t M) {
#pragma unroll
    for (int j = 0; j < Base::kN; ++j) {
      const int64_t m = mn0 + Base::row(j);
      if (m < M) {
        const int n = dHWc.div((int)m);
        const int rem = (int)m - n * (int)dHWc.d;
        const int hh = dWc.div(rem), ww = rem - hh * (int)dWc.d;
        p_[j] = hh + a;
        q_[j] = ww + b;
        base_[j] = (((int64_t)n * P + p_[j]) * Q + q_[j]) * K;
      } else {
        p_[j] = kFar;
        q_[j] = 0;
        base_[j] = 0;
      }
    }
  }
  __device__ float at(int j, int kk, int64_t kend) const {
    const bool kin = kk < kend;
    const int kc = kin ? kk : 0;
    const int i = dSK.div(kc);
    const int rem = kc - i * (int)dSK.d;
    const int jj = dK.div(rem), k = rem - jj * K;
    const bool ok = kin & inside(p_[j] - i, P) & inside(q_[j] - jj, Q);
    return *(ok ? dy + base_[j] - ((int64_t)i * Q + jj) * K + k : g_zero);
  }
  __device__ void fetch(int64_t k0, int64_t kend, float4 (&r)[Base::kN]) const {
    const int kk = (int)k0 + Base::koff();
    if constexpr (MODE == SCALAR) {
#pragma unroll
      for (int j = 0; j < Base::kN; ++j)
        r[j] = make_float4(at(j, kk, kend), at(j, kk + 1, kend), at(j, kk + 2, kend),
                           at(j, kk + 3, kend));
    } else {
      int i, jj, k;
      if constexpr (MODE == TAP) {   // uniform tap
        const int tap = dK.div((int)k0);
        i = dnS.div(tap);
        jj = tap - i * nS;
        k = (int)k0 - tap * K + Base::koff();
      } else {
        i = dSK.div(kk);
        const int rem = kk - i * (int)dSK.d;
        jj = dK.div(rem);
        k = rem - jj * K;
      }
      const int64_t toff = k - ((int64_t)i * Q + jj) * K;
      const bool kin = kk < kend;
#pragma unroll
      for (int j = 0; j < Base::kN; ++j) {
        const bool ok = kin & inside(p_[j] - i, P) & inside(q_[j] - jj, Q);
        r[j] = ld4(ok ? dy + base_[j] + toff : g_zero);
      }
    }
  }
};

// Convolution input gradient, B = filter at the class's taps:
// B[kk = (i, j, k)][c] = W[k][r0 + st i][s0 + st j][c]   (row-of-m; C % 4 == 0)
template <int E, int MODE>
struct ConvFilterTap : RowM<E> {
  using Base = RowM<E>;
  const float* w;
  int C, K, S, st, r0, s0, nS;
  int64_t RSC;
  FastDiv dK, dnS, dSK;
  int cc;                     // this lane's channel, clamped to the filter
  int64_t roff_[Base::kN];    // this lane's k rows * RSC
  __device__ void init(int64_t mn0, int64_t) {
    const int c0 = (int)mn0 + Base::moff();
    cc = c0 < C ? c0 : 0;
#pragma unroll
    for (int j = 0; j < Base::kN; ++j) roff_[j] = (int64_t)Base::krow(j) * RSC;
  }
  __device__ void fetch(int64_t k0, int64_t kend, float4 (&r)[Base::kN]) const {
    if constexpr (MODE == TAP) {   // uniform tap
      const int tap = dK.div((int)k0);
      const int i = dnS.div(tap), jj = tap - i * nS;
      const int kb = (int)k0 - tap * K;
      const float* base =
          w + (int64_t)kb * RSC + ((int64_t)(r0 + st * i) * S + s0 + st * jj) * C + cc;
#pragma unroll
      for (int j = 0; j < Base::kN; ++j) {
        const bool ok = k0 + Base::krow(j) < kend;
        r[j] = ld4(ok ? base + roff_[j] : g_zero);
      }
    } else {
#pragma unroll
      for (int j = 0; j < Base::kN; ++j) {
        const int kk = (int)k0 + Base::krow(j);
        const bool ok = kk < kend;
        const int kc = ok ? kk : 0;
        const int i = dSK.div(kc);
        const int rem = kc - i * (int)dSK.d;
        const int jj = dK.div(rem), k = rem - jj * K;
        int64_t off = (int64_t)k * RSC + ((int64_t)(r0 + st * i) * S + s0 + st * jj) * C + cc;
        keep(off);
        r[j] = ld4(ok ? w + off : g_zero);
      }
    }
  }
};

// Convolution filter gradient, B = input patches along the pixel axis:
// B[kk = (n, p, q)][col = (r, s, c)] = X[n][p st - pad + r][q st - pad + s][c]
// (row-of-m).  A lane's columns are clamped to the matrix, then split into
// taps at set-up: one tap for all of them (TAP), one per float4 (VEC4) or one
// per value (SCALAR).
template <int E, int MODE>
struct ConvPixelPatch : RowM1<E> {
  using Base = RowM1<E>;
  static constexpr int kT = MODE == TAP ? 1 : MODE == VEC4 ? Base::kN : 4 * Base::kN;
  const float* x;
  int H, W, C, st, pad;
  FastDiv dQ, dPQ, dC, dSC;
  int toff_[kT];          // (r W + s) C + c of each tap entry
  int r_[kT], s_[kT];
  __device__ void init(int64_t mn0, int64_t RSC) {
    const int col0 = (int)mn0 + Base::moff();
#pragma unroll
    for (int e = 0; e < kT; ++e) {
      const int step = MODE == VEC4 ? 4 : 1;
      const int cc = col0 + step * e < RSC ? col0 + step * e : 0;
      const int r = dSC.div(cc);
      const int rem = cc - r * (int)dSC.d;
      const int s = dC.div(rem), c = rem - s * C;
      r_[e] = r;
      s_[e] = s;
      toff_[e] = (r * W + s) * C + c;
    }
  }
  __device__ void fetch(int64_t k0, int64_t kend, float4 (&r)[Base::kN]) const {
    const int kk = (int)k0 + Base::krow();
    const bool kin = kk < kend;
    const int kc = kin ? kk : 0;
    const int n = dPQ.div(kc);
    const int rem = kc - n * (int)dPQ.d;
    const int p = dQ.div(rem), q = rem - p * (int)dQ.d;
    const int hb = p * st - pad, wb = q * st - pad;
    int64_t po = (((int64_t)n * H + hb) * W + wb) * C;
    keep(po);
    const float* pix = x + po;
    if constexpr (MODE == TAP) {
      const bool ok = kin & inside(hb + r_[0], H) & inside(wb + s_[0], W);
      const float* src = ok ? pix + toff_[0] : g_zero;
#pragma unroll
      for (int j = 0; j < Base::kN; ++j) r[j] = ld4(src + 4 * j);
    } else if constexpr (MODE == VEC4) {
#pragma unroll
      for (int j = 0; j < Base::kN; ++j) {
        const bool ok = kin & inside(hb + r_[j], H) & inside(wb + s_[j], W);
        r[j] = ld4(ok ? pix + toff_[j] : g_zero);
      }
    } else {
#pragma unroll
      for (int j = 0; j < Base::kN; ++j) {
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int u = 4 * j + e;
          const bool ok = kin & inside(hb + r_[u], H) & inside(wb + s_[u], W);
          v[e] = *(ok ? pix + toff_[u] : g_zero);
        }
        r[j] = make_float4(v[0], v[1], v[2], v[3]);
      }
    }
  }
};

// Where row m of C goes: m * ldc, or the NHWC input pixel of a stride class
struct DenseOut {
  int64_t ldc;
  __device__ int64_t row(int64_t m) const { return m * ldc; }
};
struct ClassOut {
  int H, W, C, st, ph, pw;
  FastDiv dWc, dHWc;
  __device__ int64_t row(int64_t m) const {
    const int n = dHWc.div((int)m);
    const int rem = (int)m - n * (int)dHWc.d;
    const int hh = dWc.div(rem), ww = rem - hh * (int)dWc.d;
    return (((int64_t)n * H + st * hh + ph) * W + st * ww + pw) * C;
  }
};

// ---------------------------------------------------------------- kernel
template <class L>
__device__ inline float4 read_op(const float* lds, int i, int k) {
  if (L::kRowOfK) return *reinterpret_cast<const float4*>(&lds[rowk_index(i, k)]);
  constexpr int ld = L::kLds / BK;
  return make_float4(lds[(k + 0) * ld + i], lds[(k + 1) * ld + i], lds[(k + 2) * ld + i],
                     lds[(k + 3) * ld + i]);
}

__device__ inline float comp(const float4& v, int t) {
  return t == 0 ? v.x : t == 1 ? v.y : t == 2 ? v.z : v.w;
}

// BM x BN tile; the four waves form a grid of sub-tiles made of MFMA 32 x 32
// blocks (2 x 2 waves, or 4 x 1 for tiles 32 wide and for 256 x 64 tiles, 1 x 4 for
// tiles 32 tall).
// Batched problems (grid z): batch z = (zo, zi) with zi = z mod inner; operand
// and result pointers move by zo * outer stride + zi * inner stride.  With
// skip_upper, tiles strictly above the diagonal return without writing.
struct Batch {
  int64_t inner;
  int64_t a_o, a_i, b_o, b_i, c_o, c_i;
  int64_t skip_upper;
};

template <class L>
__device__ inline void shift(L& l, int64_t d) {
  l.p += d;
}

// The wave grid of a BM x BN tile: the four waves form WM x WN, 4 x 1 for
// 32-wide and 256 x 64 tiles, 1 x 4 for 32-tall ones, else 2 x 2; each wave
// owns MB x NB MFMA 32 x 32 blocks.
template <int BM, int BN>
struct WaveGrid {
  static constexpr int WM = (BN == 32 || (BM == 256 && BN == 64)) ? 4 : BM == 32 ? 1 : 2;
  static constexpr int WN = 4 / WM;
  static constexpr int MB = BM / (32 * WM), NB = BN / (32 * WN);
  static_assert(MB >= 1 && NB >= 1 && MB * 32 * WM == BM && NB * 32 * WN == BN, "tile shape");
};

// One K tile from LDS into the accumulators: four k steps of 8 per half-wave,
// each a round of LDS reads feeding MB x NB x 4 MFMAs.
template <int BM, int BN, class LA, class LB, int MB, int NB>
__device__ __forceinline__ void mma_ktile(floatx16 (&acc)[MB][NB], const float* A, const float* B,
                                          int wm, int wn, int half, int li) {
  using G = WaveGrid<BM, BN>;
  static_assert(MB == G::MB && NB == G::NB, "accumulator blocks");
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int kq = half * 16 + 4 * j;
    float4 a[G::MB], b[G::NB];
#pragma unroll
    for (int mb = 0; mb < G::MB; ++mb) a[mb] = read_op<LA>(A, wm * (BM / G::WM) + mb * 32 + li, kq);
#pragma unroll
    for (int nb = 0; nb < G::NB; ++nb) b[nb] = read_op<LB>(B, wn * (BN / G::WN) + nb * 32 + li, kq);
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int mb = 0; mb < G::MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < G::NB; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(comp(a[mb], s), comp(b[nb], s),
                                                            acc[mb][nb], 0, 0, 0);
  }
}

// The accumulators of the tile at (m0, n0) into C (plus the column's bias).
template <int BM, int BN, class OM, bool BIAS, int MB, int NB>
__device__ __forceinline__ void store_tile(const floatx16 (&acc)[MB][NB], float* out, const OM& om,
                                           const float* bias, int64_t m0, int64_t n0, int64_t M,
                                           int64_t N, int wm, int wn, int half, int li) {
  using G = WaveGrid<BM, BN>;
  static_assert(MB == G::MB && NB == G::NB, "accumulator blocks");
#pragma unroll
  for (int mb = 0; mb < G::MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < G::NB; ++nb) {
      const int64_t col = n0 + wn * (BN / G::WN) + nb * 32 + li;
      if (col >= N) continue;
      const float bv = BIAS ? bias[col] : 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = m0 + wm * (BM / G::WM) + mb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
        if (row < M) out[om.row(row) + col] = acc[mb][nb][r] + bv;
      }
    }
}

// Issue the next tile's global loads one per two MFMAs from the start of a K
// tile's body, so that the MFMAs cover their latency; left alone, the
// scheduler sinks them next to the LDS stores that consume them.
template <int NLOADS>
__device__ __forceinline__ void interleave_loads() {
#pragma unroll
  for (int g = 0; g < NLOADS; ++g) {
    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // one global load
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);   // two MFMAs
  }
}

// ROWSUM: rowsum[slice][m] = sum over this slice's k of A[m][k]
template <int BM, int BN, class LA, class LB, class OM, bool BIAS, bool BATCHED, bool ROWSUM>
__global__ __launch_bounds__(THREADS) void gemm_kernel(LA la, LB lb, float* __restrict__ c, OM om,
                                                       int64_t slice_stride,
                                                       const float* __restrict__ bias, int64_t M,
                                                       int64_t N, int64_t K, int64_t k_slice,
                                                       int tiles_m, int tiles_n, Batch bt,
                                                       float* __restrict__ rowsum) {
  constexpr int WM = WaveGrid<BM, BN>::WM, MB = WaveGrid<BM, BN>::MB, NB = WaveGrid<BM, BN>::NB;
  constexpr bool kLoadsFirst = BN > 128;
  // Workgroup (tile, slice, batch) from an XCD-aware order: the hardware hands
  // linear workgroup h to XCD h mod 8, so logical ids are laid out so that each
  // XCD (with its own L2) gets one contiguous run of them, and neighbouring
  // tiles, which share operand rows, share an L2.
  const uint32_t gx = gridDim.x, gy = gridDim.y;
  const uint32_t G = gx * gy * gridDim.z;
  const uint32_t h = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
  const uint32_t q = G / kXcds, rem = G % kXcds, xcd = h % kXcds, local = h / kXcds;
  const uint32_t L = xcd < rem ? xcd * (q + 1) + local : rem * (q + 1) + (xcd - rem) * q + local;
  const int t = (int)(L % gx);
  const int64_t slice = (L / gx) % gy;
  if constexpr (BATCHED) {
    const int64_t z = L / (gx * gy), zo = z / bt.inner, zi = z % bt.inner;
    shift(la, zo * bt.a_o + zi * bt.a_i);
    shift(lb, zo * bt.b_o + zi * bt.b_i);
    c += zo * bt.c_o + zi * bt.c_i;
  }
  __shared__ __attribute__((aligned(16))) float As[2][LA::kLds];
  __shared__ __attribute__((aligned(16))) float Bs[2][LB::kLds];

  // grouped tile order: 8 tile-rows share their B tiles in L2
  const int group = 8;
  const int per_group = group * tiles_n;
  const int g = t / per_group;
  const int first_m = g * group;
  const int gsize = min(tiles_m - first_m, group);
  const int tm = first_m + (t % per_group) % gsize;
  const int tn = (t % per_group) / gsize;
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  if constexpr (BATCHED) {
    if (bt.skip_upper && n0 >= m0 + BM) return;   // the whole workgroup leaves together
  }
  const int64_t kb = slice * k_slice;
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

  const bool sums = ROWSUM && tn == 0 && (int)threadIdx.x < BM;
  float rs = 0.f;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave % WM, wn = wave / WM;
  const int half = lane >> 5;
  const int li = lane & 31;

  la.fetch(kb, ke, ra);
  lb.fetch(kb, ke, rb);
  LA::store(As[0], ra);
  LB::store(Bs[0], rb);
  __syncthreads();
  int buf = 0;
  for (int64_t k0 = kb; k0 < ke; k0 += BK) {
    // the tile after the last one is all zeros: fetching and storing it anyway
    // keeps the loop body free of branches
    la.fetch(k0 + BK, ke, ra);
    lb.fetch(k0 + BK, ke, rb);
    // 192-wide tiles issue all their loads before the MFMAs: their address
    // arithmetic is long enough that the interleave below would place the
    // loads late (measured 2-4 % slower)
    if constexpr (kLoadsFirst) __builtin_amdgcn_sched_barrier(0);
    const float* A = As[buf];
    const float* B = Bs[buf];
    mma_ktile<BM, BN, LA, LB>(acc, A, B, wm, wn, half, li);
    if constexpr (ROWSUM) {
      if (sums) {
#pragma unroll
        for (int k = 0; k < BK; ++k) {
          if constexpr (LA::kRowOfK) rs += A[rowk_index(threadIdx.x, k)];
          else rs += A[k * (LA::kLds / BK) + threadIdx.x];
        }
      }
    }
    if constexpr (!kLoadsFirst) interleave_loads<LA::kN + LB::kN>();
    LA::store(As[buf ^ 1], ra);
    LB::store(Bs[buf ^ 1], rb);
    __syncthreads();
    buf ^= 1;
  }

  if (sums && m0 + threadIdx.x < M) rowsum[slice * M + m0 + threadIdx.x] = rs;
  store_tile<BM, BN, OM, BIAS>(acc, c + slice * slice_stride, om, bias, m0, n0, M, N, wm, wn, half,
                               li);
}

// Persistent form for short reductions of the dense loaders (one slice, no
// batch, no row sums; chosen below): a workgroup walks the tiles L, L + G,
// L + 2G, ... and, while it multiplies the last K tile of one output tile,
// already loads the first K tile of its next one, so that the next tile's
// loads and this tile's stores are in flight together.  With K of 64 or 128 a
// tile has only two or four K tiles, and the one-tile-per-workgroup form spends
// much of each workgroup's life in its first load and its stores.  Results are
// those of gemm_kernel bit for bit (same K order per output).
template <int BM, int BN, class LA, class LB, class OM, bool BIAS>
__global__ __launch_bounds__(THREADS) void gemm_persistent(LA la, LB lb, float* __restrict__ c,
                                                           OM om, const float* __restrict__ bias,
                                                           int64_t M, int64_t N, int64_t K,
                                                           int tiles_m, int tiles_n) {
  constexpr int WM = WaveGrid<BM, BN>::WM, MB = WaveGrid<BM, BN>::MB, NB = WaveGrid<BM, BN>::NB;
  static_assert(BN <= 128, "loads interleaved with the MFMAs, as gemm_kernel does up to 128 wide");
  // the same XCD-aware logical order as gemm_kernel: each XCD's workgroups take
  // one contiguous run of tiles in every round
  const uint32_t G = gridDim.x, h = blockIdx.x;
  const uint32_t q = G / kXcds, rem = G % kXcds, xcd = h % kXcds, local = h / kXcds;
  const uint32_t L = xcd < rem ? xcd * (q + 1) + local : rem * (q + 1) + (xcd - rem) * q + local;
  const int n_tiles = tiles_m * tiles_n;
  int t = (int)L;
  if (t >= n_tiles) return;   // the whole workgroup leaves together
  __shared__ __attribute__((aligned(16))) float As[2][LA::kLds];
  __shared__ __attribute__((aligned(16))) float Bs[2][LB::kLds];
  const int group = 8;        // grouped tile order, as in gemm_kernel
  const int per_group = group * tiles_n;
  auto origin = [&](int tt, int64_t& m0, int64_t& n0) {
    const int g = tt / per_group;
    const int first_m = g * group;
    const int gsize = min(tiles_m - first_m, group);
    m0 = (int64_t)(first_m + (tt % per_group) % gsize) * BM;
    n0 = (int64_t)((tt % per_group) / gsize) * BN;
  };
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wm = wave % WM, wn = wave / WM;
  const int half = lane >> 5;
  const int li = lane & 31;
  int64_t m0, n0;
  origin(t, m0, n0);
  la.init(m0, M);
  lb.init(n0, N);
  float4 ra[LA::kN], rb[LB::kN];
  la.fetch(0, K, ra);
  lb.fetch(0, K, rb);
  LA::store(As[0], ra);
  LB::store(Bs[0], rb);
  __syncthreads();
  int buf = 0;
  while (true) {
    floatx16 acc[MB][NB];
#pragma unroll
    for (int a = 0; a < MB; ++a)
#pragma unroll
      for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;
    for (int64_t k0 = 0; k0 + BK < K; k0 += BK) {
      la.fetch(k0 + BK, K, ra);
      lb.fetch(k0 + BK, K, rb);
      mma_ktile<BM, BN, LA, LB>(acc, As[buf], Bs[buf], wm, wn, half, li);
      interleave_loads<LA::kN + LB::kN>();
      LA::store(As[buf ^ 1], ra);
      LB::store(Bs[buf ^ 1], rb);
      __syncthreads();
      buf ^= 1;
    }
    // the last K tile; the next output tile's first K tile is loaded meanwhile
    // into the other buffer, which no wave reads until the barrier below
    const int tn = t + (int)G;
    const bool more = tn < n_tiles;   // uniform over the workgroup
    int64_t m1 = 0, n1 = 0;
    if (more) {
      origin(tn, m1, n1);
      la.init(m1, M);
      lb.init(n1, N);
      la.fetch(0, K, ra);
      lb.fetch(0, K, rb);
    }
    mma_ktile<BM, BN, LA, LB>(acc, As[buf], Bs[buf], wm, wn, half, li);
    if (more) {
      LA::store(As[buf ^ 1], ra);
      LB::store(Bs[buf ^ 1], rb);
    }
    store_tile<BM, BN, OM, BIAS>(acc, c, om, bias, m0, n0, M, N, wm, wn, half, li);
    if (!more) break;
    __syncthreads();
    buf ^= 1;
    t = tn;
    m0 = m1;
    n0 = n1;
  }
}

// Loaders the persistent form is used with: the plain matrix views.
template <class L> struct DenseView : std::false_type {};
template <int E, bool V> struct DenseView<MatK<E, V>> : std::true_type {};
template <int E, bool V> struct DenseView<MatM<E, V>> : std::true_type {};
constexpr int64_t kShortK = 128;   // reductions at most this long run persistent

template <int BM, int BN, class LA, class LB, class OM, bool BIAS, bool BATCHED = false,
          bool ROWSUM = false>
hipError_t run_gemm(const LA& la, const LB& lb, float* c, OM om, int64_t slice_stride,
                    const float* bias, int64_t M, int64_t N, int64_t K, int64_t slices,
                    hipStream_t s, int64_t batches = 1, Batch bt = Batch{1, 0, 0, 0, 0, 0, 0, 0},
                    float* rowsum = nullptr) {
  const int64_t tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  if (tiles_m * tiles_n > INT32_MAX / 2 || slices > 65535 || batches > 65535 || batches < 1 ||
      tiles_m * tiles_n * slices * batches > INT32_MAX)
    return hipErrorInvalidValue;
  int64_t k_slice = (K + slices - 1) / slices;
  k_slice = (k_slice + BK - 1) / BK * BK;
  if (ROWSUM != (rowsum != nullptr)) return hipErrorInvalidValue;
  if constexpr (!BATCHED && !ROWSUM && DenseView<LA>::value && DenseView<LB>::value) {
    if (slices == 1 && K <= kShortK) {
      // one workgroup per resident slot (the occupancy query counts LDS and registers)
      auto kern = gemm_persistent<BM, BN, LA, LB, OM, BIAS>;
      static const int64_t slots = [&] {   // initialised once, thread-safe
        int o = 0, n = 0, dev = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&o, kern, THREADS, 0) != hipSuccess ||
            o < 1)
          o = 1;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            n < 1)
          n = 256;
        return (int64_t)o * n;
      }();
      const int64_t G = std::min<int64_t>(tiles_m * tiles_n, slots);
      hipLaunchKernelGGL(kern, dim3((unsigned)G), dim3(THREADS), 0, s, la, lb, c, om, bias, M, N,
                         K, (int)tiles_m, (int)tiles_n);
      return hipGetLastError();
    }
  }
  dim3 grid((unsigned)(tiles_m * tiles_n), (unsigned)slices, (unsigned)batches);
  hipLaunchKernelGGL((gemm_kernel<BM, BN, LA, LB, OM, BIAS, BATCHED, ROWSUM>), grid, dim3(THREADS), 0, s,
                     la, lb, c, om, slice_stride, bias, M, N, K, k_slice, (int)tiles_m,
                     (int)tiles_n, bt, rowsum);
  return hipGetLastError();
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// Tile shape: 128 x 128, or 64 along a dimension that is at most 64 wide
// (half of a 128-wide tile would compute zeros).  At most 64 columns and many
// rows (the 64-channel convolutions) take 256 x 64: each wave then owns 64 x 64
// and one round of LDS reads feeds 16 MFMAs instead of 8 (2-3 % faster
// measured; plain, unbatched products only, to keep the kernel count down).
// A product with fewer 128 x 128 tiles than half the CUs and a reduction of at
// most 4096 (a dense layer at a small batch) takes 64 x 64 tiles, four times
// as many workgroups, each wave one MFMA block.  Longer reductions keep
// 128 x 128: those of few tiles are weight gradients, which split their rows
// into slices instead.  Unbatched products only: a batched product has
// workgroups enough across its batch.
constexpr int64_t kTallRows = 65536;
constexpr int64_t kFewTiles = 128;
constexpr int64_t kFewTilesMaxK = 4096;
enum Shape { S128x128, S128x64, S64x128, S256x64, S64x64 };
Shape pick_shape(int64_t M, int64_t N, int64_t K) {
  if (N <= 64 && M >= kTallRows) return S256x64;
  if (N <= 64 && M > 64) return S128x64;
  if (M <= 64) return S64x128;
  if (((M + 127) / 128) * ((N + 127) / 128) < kFewTiles && K <= kFewTilesMaxK) return S64x64;
  return S128x128;
}

// Runs the GEMM with loader templates A<E>, B<E> instantiated for the chosen
// tile shape; `fa(a)` / `fb(b)` fill them in.  Row m of C starts at om.row(m);
// split-K slices of C are slice_stride floats apart.
template <template <int> class LAT, template <int> class LBT, bool BIAS, bool BATCHED = false,
          bool ROWSUM = false, class FA, class FB, class OM>
hipError_t dispatch(FA fa, FB fb, float* c, OM om, int64_t slice_stride, const float* bias,
                    int64_t M, int64_t N, int64_t K, int64_t slices, hipStream_t s,
                    int64_t batches = 1, Batch bt = Batch{1, 0, 0, 0, 0, 0, 0, 0},
                    float* rowsum = nullptr) {
  switch (pick_shape(M, N, K)) {
    case S256x64:
      if constexpr (!BATCHED && !ROWSUM) {
        LAT<256> a{};
        LBT<64> b{};
        fa(a);
        fb(b);
        return run_gemm<256, 64, LAT<256>, LBT<64>, OM, BIAS, false, false>(
            a, b, c, om, slice_stride, bias, M, N, K, slices, s);
      }
      [[fallthrough]];
    case S128x64: {
      LAT<128> a{};
      LBT<64> b{};
      fa(a);
      fb(b);
      return run_gemm<128, 64, LAT<128>, LBT<64>, OM, BIAS, BATCHED, ROWSUM>(
          a, b, c, om, slice_stride, bias, M, N, K, slices, s, batches, bt, rowsum);
    }
    case S64x128: {
      LAT<64> a{};
      LBT<128> b{};
      fa(a);
      fb(b);
      return run_gemm<64, 128, LAT<64>, LBT<128>, OM, BIAS, BATCHED, ROWSUM>(
          a, b, c, om, slice_stride, bias, M, N, K, slices, s, batches, bt, rowsum);
    }
    case S64x64:
      if constexpr (!BATCHED) {
        LAT<64> a{};
        LBT<64> b{};
        fa(a);
        fb(b);
        return run_gemm<64, 64, LAT<64>, LBT<64>, OM, BIAS, false, ROWSUM>(
            a, b, c, om, slice_stride, bias, M, N, K, slices, s, 1, bt, rowsum);
      }
      [[fallthrough]];
    default: {
      LAT<128> a{};
      LBT<128> b{};
      fa(a);
      fb(b);
      return run_gemm<128, 128, LAT<128>, LBT<128>, OM, BIAS, BATCHED, ROWSUM>(
          a, b, c, om, slice_stride, bias, M, N, K, slices, s, batches, bt, rowsum);
    }
  }
}

// row-major C with leading dimension ldc
template <template <int> class LAT, template <int> class LBT, bool BIAS, bool BATCHED = false,
          bool ROWSUM = false, class FA, class FB>
hipError_t dispatch_dense(FA fa, FB fb, float* c, int64_t ldc, const float* bias, int64_t M,
                          int64_t N, int64_t K, int64_t slices, hipStream_t s,
                          int64_t batches = 1, Batch bt = Batch{1, 0, 0, 0, 0, 0, 0, 0},
                          float* rowsum = nullptr) {
  return dispatch<LAT, LBT, BIAS, BATCHED, ROWSUM>(fa, fb, c, DenseOut{ldc}, M * ldc, bias, M, N, K,
                                                   slices, s, batches, bt, rowsum);
}

// one explicit tile shape, loaders instantiated at its extents
template <int BM, int BN, template <int> class LAT, template <int> class LBT, class FA, class FB,
          class OM>
hipError_t dispatch_shape(FA fa, FB fb, float* c, OM om, int64_t slice_stride, int64_t M,
                          int64_t N, int64_t K, int64_t slices, hipStream_t s) {
  LAT<BM> a{};
  LBT<BN> b{};
  fa(a);
  fb(b);
  return run_gemm<BM, BN, LAT<BM>, LBT<BN>, OM, false>(a, b, c, om, slice_stride, nullptr, M, N, K,
                                                       slices, s);
}

template <int E> using MatKv = MatK<E, true>;
template <int E> using MatKs = MatK<E, false>;
template <int E> using MatMv = MatM<E, true>;
template <int E> using MatMs = MatM<E, false>;
template <int E> using ConvPatchT = ConvPatch<E, TAP>;
template <int E> using ConvPatchV = ConvPatch<E, VEC4>;
template <int E> using ConvPatchS = ConvPatch<E, SCALAR>;
template <int E> using ConvGradTapT = ConvGradTap<E, TAP>;
template <int E> using ConvGradTapV = ConvGradTap<E, VEC4>;
template <int E> using ConvGradTapS = ConvGradTap<E, SCALAR>;
template <int E> using ConvFilterTapT = ConvFilterTap<E, TAP>;
template <int E> using ConvFilterTapG = ConvFilterTap<E, VEC4>;
template <int E> using ConvPixelPatchT = ConvPixelPatch<E, TAP>;
template <int E> using ConvPixelPatchV = ConvPixelPatch<E, VEC4>;
template <int E> using ConvPixelPatchS = ConvPixelPatch<E, SCALAR>;

// the GEMM sizes of the convolution views index with 32-bit arithmetic
bool fits31(int64_t v) { return v >= 0 && v < (int64_t(1) << 31) - 64; }

// Tile of a filter gradient (M = output channels, N = RSC), first rule that
// applies; the lowering's split-K slice count follows the same rule:
//   32 x 256 for M <= 32 (no empty tile rows; 32 columns of one tap a thread
//            when C % 32 == 0);
//   64 x 192 for M <= 64 when that leaves fewer padded RSC columns than
//            64 x 128 (RSC = 576 for a 3 x 3 x 64 filter: 3 full tiles, not 4.5);
//   64 x 64  for M <= 64 and RSC <= 64 (1 x 1 filters, 3-channel inputs);
//   otherwise the general shapes.
// The first three need M % 4 == 0 (and C % 4 == 0 for the first two).
enum class WgradTile { k32x256, k64x192, k64x64, kGeneral };
WgradTile wgrad_tile(int64_t M, int64_t N, int64_t C) {
  if (M % 4 != 0) return WgradTile::kGeneral;
  if (M <= 32 && C % 4 == 0) return WgradTile::k32x256;
  const int64_t pad128 = (N + 127) / 128 * 128 - N, pad192 = (N + 191) / 192 * 192 - N;
  if (M <= 64 && C % 4 == 0 && pad192 < pad128) return WgradTile::k64x192;
  if (M <= 64 && N <= 64) return WgradTile::k64x64;
  return WgradTile::kGeneral;
}

// ---------------------------------------------------------------- small kernels
// out[j] = sum over slices of part[s][j].  A workgroup covers 64 consecutive
// j, one per lane; wave w takes the slices s = w mod 4 in eight interleaved
// chains (s / 4 mod 8), so that each lane has eight loads in flight, and the
// partial sums are added in a fixed order: the result does not depend on
// timing.
constexpr int SUM_J = 64;
__global__ __launch_bounds__(256) void slice_sum_kernel(const float* __restrict__ part,
                                                        float* __restrict__ out, int64_t n,
                                                        int64_t slices) {
  __shared__ float red[4][SUM_J];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t j = (int64_t)blockIdx.x * SUM_J + lane;
  float a[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (j < n) {
    int64_t s = w;
    for (; s + 28 < slices; s += 32) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = part[(s + 4 * u) * n + j];
#pragma unroll
      for (int u = 0; u < 8; ++u) a[u] += v[u];
    }
#pragma unroll
    for (int u = 0; u < 7; ++u)
      if (s + 4 * u < slices) a[u] += part[(s + 4 * u) * n + j];
  }
  red[w][lane] = ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]));
  __syncthreads();
  if (w == 0 && j < n) out[j] = (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]);
}

hipError_t slice_sum(const float* part, float* out, int64_t n, int64_t slices, hipStream_t s) {
  hipLaunchKernelGGL(slice_sum_kernel, dim3((unsigned)((n + SUM_J - 1) / SUM_J)), dim3(256), 0, s,
                     part, out, n, slices);
  return hipGetLastError();
}

// The input-gradient pixels of a stride class that no filter tap reaches are
// zeros (a 1 x 1 filter with stride 2 reaches one class of four).  Rows
// m0 .. m0 + rows of the class, q = C / 4 float4 each; rows * q < 2^31.
__global__ __launch_bounds__(256) void class_zero_kernel(float* __restrict__ dx, ClassOut om,
                                                         int64_t m0, int rows, int q,
                                                         FastDiv dq) {
  const int n = rows * q;
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) {
    const int r = dq.div(i);
    *reinterpret_cast<float4*>(dx + om.row(m0 + r) + 4 * (i - r * q)) = make_float4(0, 0, 0, 0);
  }
}

hipError_t class_zero(float* dx, const ClassOut& om, int64_t M, int64_t C, hipStream_t s) {
  const int64_t q = C / 4;
  const int64_t per = std::max<int64_t>(1, (int64_t(1) << 30) / q);   // rows per launch
  for (int64_t m0 = 0; m0 < M; m0 += per) {
    const int64_t rows = std::min(per, M - m0);
    const int64_t blocks = std::min<int64_t>((rows * q + 255) / 256, 16384);
    hipLaunchKernelGGL(class_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, s, dx, om, m0,
                       (int)rows, (int)q, FastDiv::make(q));
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace

// ---------------------------------------------------------------- launchers
hipError_t linear_fwd(const float* X, const float* W, const float* b, float* Y, int64_t M,
                      int64_t K, int64_t N, hipStream_t s) {
  auto fa = [&](auto& a) { a.p = X; a.ld = K; };
  auto fb = [&](auto& bb) { bb.p = W; bb.ld = K; };
  if (K % 4 == 0 && aligned16(X) && aligned16(W))
    return dispatch_dense<MatKv, MatKv, true>(fa, fb, Y, N, b, M, N, K, 1, s);
  return dispatch_dense<MatKs, MatKs, true>(fa, fb, Y, N, b, M, N, K, 1, s);
}

hipError_t linear_bwd_x(const float* W, const float* dY, float* dX, int64_t M, int64_t K,
                        int64_t N, hipStream_t s) {
  // dX[M][K] = dY[M][N] W[N][K]: A = dY (contiguous along the reduction), B[n_out][k_in] = W
  auto fa = [&](auto& a) { a.p = dY; a.ld = N; };
  auto fb = [&](auto& bb) { bb.p = W; bb.ld = K; };
  if (N % 4 == 0 && K % 4 == 0 && aligned16(W) && aligned16(dY))
    return dispatch_dense<MatKv, MatMv, false>(fa, fb, dX, K, nullptr, M, K, N, 1, s);
  return dispatch_dense<MatKs, MatMs, false>(fa, fb, dX, K, nullptr, M, K, N, 1, s);
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
    e = dispatch_dense<MatMv, MatMv, false, false, true>(fa, fb, out, K, nullptr, N, K, M, slices,
                                                         s, 1, one, sums);
  else
    e = dispatch_dense<MatMs, MatMs, false, false, true>(fa, fb, out, K, nullptr, N, K, M, slices,
                                                         s, 1, one, sums);
  if (e != hipSuccess || slices <= 1) return e;
  e = slice_sum(part, dW, N * K, slices, s);
  if (e != hipSuccess) return e;
  return slice_sum(sums, db, N, slices, s);
}

hipError_t gemm_batched(bool a_rowk, const float* A, int64_t lda, bool b_rowk, const float* B,
                        int64_t ldb, float* C, int64_t ldc, int64_t M, int64_t N, int64_t K,
                        int64_t batches, const BatchStrides& st, hipStream_t s) {
  const Batch bt{st.inner,   st.a_outer, st.a_inner, st.b_outer,
                 st.b_inner, st.c_outer, st.c_inner, st.skip_upper};
  auto fa = [&](auto& a) { a.p = A; a.ld = lda; };
  auto fb = [&](auto& b) { b.p = B; b.ld = ldb; };
  const bool vec = lda % 4 == 0 && ldb % 4 == 0 && aligned16(A) && aligned16(B) &&
                   (a_rowk ? K % 4 == 0 : M % 4 == 0) && (b_rowk ? K % 4 == 0 : N % 4 == 0) &&
                   st.a_outer % 4 == 0 && st.a_inner % 4 == 0 && st.b_outer % 4 == 0 &&
                   st.b_inner % 4 == 0;
#define GEMM_BATCHED_CASE(LA, LB) \
  return dispatch_dense<LA, LB, false, true>(fa, fb, C, ldc, nullptr, M, N, K, 1, s, batches, bt)
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

// A 1 x 1 convolution with stride 1 and no padding is a plain product of the
// NHWC pixel rows: its forward is X W^T, its input gradient dY W and its filter
// gradient dY^T X, all run on the dense loaders (one add per K tile for the
// address, no tap arithmetic).
static bool pointwise(const ConvShape& c) {
  return c.R == 1 && c.S == 1 && c.stride == 1 && c.pad == 0 && c.C % 4 == 0 && c.K % 4 == 0;
}

hipError_t conv_fwd(const float* X, const float* W, float* Y, const ConvShape& c, hipStream_t s) {
  const int64_t M = c.N * c.P * c.Q, N = c.K, K = c.R * c.S * c.C;
  if (!fits31(M) || !fits31(K)) return hipErrorInvalidValue;
  if (pointwise(c) && N > 32 && aligned16(X) && aligned16(W)) {
    // Y[NPQ][K] = X[NPQ][C] W[K][C]^T
    auto fa = [&](auto& a) { a.p = X; a.ld = c.C; };
    auto fb = [&](auto& b) { b.p = W; b.ld = c.C; };
    return dispatch_dense<MatKv, MatKv, false>(fa, fb, Y, N, nullptr, M, N, K, 1, s);
  }
  auto fa = [&](auto& a) {
    a.x = X; a.H = (int)c.H; a.W = (int)c.W; a.C = (int)c.C; a.S = (int)c.S;
    a.st = (int)c.stride; a.pad = (int)c.pad;
    a.dQ = FastDiv::make(c.Q); a.dPQ = FastDiv::make(c.P * c.Q); a.dC = FastDiv::make(c.C);
    a.dS = FastDiv::make(c.S); a.dSC = FastDiv::make(c.S * c.C);
  };
  auto fb = [&](auto& b) { b.p = W; b.ld = K; };
  if (N <= 32 && c.C % 4 == 0) {
    // at most 32 output channels: 256 x 32 tiles, no empty columns; 128 x 32 when there are
    // fewer 256-row tiles than CUs, so that twice as many workgroups share the chip
    if ((M + 255) / 256 < 256) {
      if (c.C % 32 == 0)
        return dispatch_shape<128, 32, ConvPatchT, MatKv>(fa, fb, Y, DenseOut{N}, 0, M, N, K, 1, s);
      return dispatch_shape<128, 32, ConvPatchV, MatKv>(fa, fb, Y, DenseOut{N}, 0, M, N, K, 1, s);
    }
    if (c.C % 32 == 0)
      return dispatch_shape<256, 32, ConvPatchT, MatKv>(fa, fb, Y, DenseOut{N}, 0, M, N, K, 1, s);
    return dispatch_shape<256, 32, ConvPatchV, MatKv>(fa, fb, Y, DenseOut{N}, 0, M, N, K, 1, s);
  }
  if (c.C % 32 == 0)
    return dispatch_dense<ConvPatchT, MatKv, false>(fa, fb, Y, N, nullptr, M, N, K, 1, s);
  if (c.C % 4 == 0)
    return dispatch_dense<ConvPatchV, MatKv, false>(fa, fb, Y, N, nullptr, M, N, K, 1, s);
  return dispatch_dense<ConvPatchS, MatKs, false>(fa, fb, Y, N, nullptr, M, N, K, 1, s);
}

hipError_t conv_bwd_x(const float* W, const float* dY, float* dX, const ConvShape& c,
                      hipStream_t s) {
  if (c.C % 4 != 0) return hipErrorInvalidValue;   // every conv with an input gradient has C % 4 == 0
  if (!fits31(c.N * c.H * c.W) || !fits31(c.R * c.S * c.K)) return hipErrorInvalidValue;
  if (pointwise(c) && aligned16(W) && aligned16(dY)) {
    // dX[NHW][C] = dY[NHW][K] W[K][C]
    auto fa = [&](auto& a) { a.p = dY; a.ld = c.K; };
    auto fb = [&](auto& b) { b.p = W; b.ld = c.C; };
    return dispatch_dense<MatKv, MatMv, false>(fa, fb, dX, c.C, nullptr, c.N * c.H * c.W, c.C, c.K,
                                               1, s);
  }
  const int64_t st = c.stride;
  // one GEMM per stride class (ph, pw) of input pixels; a class no tap reaches gets zeros
  for (int64_t ph = 0; ph < st; ++ph)
    for (int64_t pw = 0; pw < st; ++pw) {
      const int64_t Hc = (c.H - ph + st - 1) / st, Wc = (c.W - pw + st - 1) / st;
      const int64_t r0 = (ph + c.pad) % st, s0 = (pw + c.pad) % st;
      const int64_t nR = r0 < c.R ? (c.R - r0 + st - 1) / st : 0;
      const int64_t nS = s0 < c.S ? (c.S - s0 + st - 1) / st : 0;
      const int64_t M = c.N * Hc * Wc, N = c.C, K = nR * nS * c.K;
      if (M == 0) continue;
      auto fa = [&](auto& a) {
        a.dy = dY; a.P = (int)c.P; a.Q = (int)c.Q; a.K = (int)c.K; a.nS = (int)nS;
        a.a = (int)((ph + c.pad - r0) / st); a.b = (int)((pw + c.pad - s0) / st);
        a.dWc = FastDiv::make(Wc); a.dHWc = FastDiv::make(Hc * Wc); a.dK = FastDiv::make(c.K);
        a.dnS = FastDiv::make(nS > 0 ? nS : 1); a.dSK = FastDiv::make(nS > 0 ? nS * c.K : 1);
      };
      auto fb = [&](auto& b) {
        b.w = W; b.C = (int)c.C; b.K = (int)c.K; b.S = (int)c.S; b.st = (int)st; b.r0 = (int)r0;
        b.s0 = (int)s0; b.nS = (int)nS; b.RSC = c.R * c.S * c.C;
        b.dK = FastDiv::make(c.K); b.dnS = FastDiv::make(nS > 0 ? nS : 1);
        b.dSK = FastDiv::make(nS > 0 ? nS * c.K : 1);
      };
      const ClassOut om{(int)c.H, (int)c.W, (int)c.C, (int)st, (int)ph, (int)pw,
                        FastDiv::make(Wc), FastDiv::make(Hc * Wc)};
      hipError_t e;
      if (K == 0 && aligned16(dX))   // no tap: a plain fill instead of an empty product
        e = class_zero(dX, om, M, c.C, s);
      else if (c.K % 32 == 0)
        e = dispatch<ConvGradTapT, ConvFilterTapT, false>(fa, fb, dX, om, 0, nullptr, M, N, K, 1,
                                                          s);
      else if (c.K % 4 == 0)
        e = dispatch<ConvGradTapV, ConvFilterTapG, false>(fa, fb, dX, om, 0, nullptr, M, N, K, 1,
                                                          s);
      else
        e = dispatch<ConvGradTapS, ConvFilterTapG, false>(fa, fb, dX, om, 0, nullptr, M, N, K, 1,
                                                          s);
      if (e != hipSuccess) return e;
    }
  return hipSuccess;
}

hipError_t conv_bwd_w(const float* X, const float* dY, float* dW, float* part, int64_t slices,
                      const ConvShape& c, hipStream_t s) {
  // dW[K][RSC] = sum over pixels of dY[pixel][k] * patch[pixel][rsc]
  const int64_t M = c.K, N = c.R * c.S * c.C, K = c.N * c.P * c.Q;
  if (!fits31(K) || !fits31(N) || !fits31((c.R * c.W + c.S) * c.C)) return hipErrorInvalidValue;
  if (slices > 1 && part == nullptr) return hipErrorInvalidValue;
  float* out = slices > 1 ? part : dW;
  auto fa = [&](auto& a) { a.p = dY; a.ld = c.K; };
  auto fb = [&](auto& b) {
    b.x = X; b.H = (int)c.H; b.W = (int)c.W; b.C = (int)c.C; b.st = (int)c.stride;
    b.pad = (int)c.pad; b.dQ = FastDiv::make(c.Q); b.dPQ = FastDiv::make(c.P * c.Q);
    b.dC = FastDiv::make(c.C); b.dSC = FastDiv::make(c.S * c.C);
  };
  const DenseOut om{N};
  hipError_t e;
  switch (wgrad_tile(M, N, c.C)) {
    case WgradTile::k32x256:   // at most 32 output channels: no empty tile rows
      e = c.C % 32 == 0
              ? dispatch_shape<32, 256, MatMv, ConvPixelPatchT>(fa, fb, out, om, M * N, M, N, K,
                                                                slices, s)
              : dispatch_shape<32, 256, MatMv, ConvPixelPatchV>(fa, fb, out, om, M * N, M, N, K,
                                                                slices, s);
      break;
    case WgradTile::k64x192:   // no tile column half empty when RSC is an odd multiple of 64
      e = dispatch_shape<64, 192, MatMv, ConvPixelPatchV>(fa, fb, out, om, M * N, M, N, K, slices,
                                                          s);
      break;
    case WgradTile::k64x64:    // RSC of at most 64 (1 x 1 filters, the 3-channel first layer)
      e = c.C % 16 == 0 ? dispatch_shape<64, 64, MatMv, ConvPixelPatchT>(fa, fb, out, om, M * N, M,
                                                                         N, K, slices, s)
          : c.C % 4 == 0 ? dispatch_shape<64, 64, MatMv, ConvPixelPatchV>(fa, fb, out, om, M * N,
                                                                          M, N, K, slices, s)
                         : dispatch_shape<64, 64, MatMv, ConvPixelPatchS>(fa, fb, out, om, M * N,
                                                                          M, N, K, slices, s);
      break;
    default:
      if (pointwise(c) && aligned16(X) && aligned16(dY)) {
        // dW[K][C] = dY^T X over the pixel rows: the dense weight gradient's loaders (the same
        // tile shapes as the general case below, so the slice count is the same)
        auto fx = [&](auto& b) { b.p = X; b.ld = c.C; };
        e = dispatch_dense<MatMv, MatMv, false>(fa, fx, out, N, nullptr, M, N, K, slices, s);
      } else if (c.K % 4 != 0)
        e = dispatch_dense<MatMs, ConvPixelPatchS, false>(fa, fb, out, N, nullptr, M, N, K, slices,
                                                          s);
      else if (c.C % 16 == 0)
        e = dispatch_dense<MatMv, ConvPixelPatchT, false>(fa, fb, out, N, nullptr, M, N, K, slices,
                                                          s);
      else if (c.C % 4 == 0)
        e = dispatch_dense<MatMv, ConvPixelPatchV, false>(fa, fb, out, N, nullptr, M, N, K, slices,
                                                          s);
      else
        e = dispatch_dense<MatMv, ConvPixelPatchS, false>(fa, fb, out, N, nullptr, M, N, K, slices,
                                                          s);
  }
  if (e != hipSuccess || slices <= 1) return e;
  return slice_sum(part, dW, M * N, slices, s);
}

// Split-K slice count of a weight gradient with M x N outputs reduced over K
// rows (C = input channels of a filter gradient, -1 for a dense layer).  The
// launchers above run tiles x s workgroups; a CU holds kResident of them at
// once (LDS bounds it: 2 for 128 x 128, 64 x 192 and 32 x 256 tiles, 3 for the
// general 64-wide ones, 4-5 for the 64 x 64 tiles), so a launch
// takes ceil(tiles s / slots) rounds of K / s rows.  s minimises rounds / s
// (a partly filled last round leaves most CUs idle behind a few), with at most
// four rounds and at least 256 rows a slice; the smallest s within 1 % of the
// best is taken, since every slice adds one partial dW to write and read back.
int64_t wgrad_slices(int64_t M, int64_t N, int64_t K, int64_t C) {
  constexpr int64_t kCUs = 256;
  int64_t tiles, resident;
  const WgradTile t = C >= 0 ? wgrad_tile(M, N, C) : WgradTile::kGeneral;
  if (t == WgradTile::k32x256) {
    tiles = (N + 255) / 256, resident = 2;
  } else if (t == WgradTile::k64x192) {
    tiles = (N + 191) / 192, resident = 2;
  } else if (t == WgradTile::k64x64) {
    tiles = 1, resident = C % 4 == 0 ? 5 : 4;
  } else {
    switch (pick_shape(M, N, K)) {
      case S256x64: tiles = (M + 255) / 256, resident = 2; break;
      case S128x64: tiles = (M + 127) / 128, resident = 3; break;
      case S64x128: tiles = (N + 127) / 128, resident = 3; break;
      case S64x64: tiles = ((M + 63) / 64) * ((N + 63) / 64), resident = 4; break;
      default: tiles = ((M + 127) / 128) * ((N + 127) / 128), resident = 2;
    }
  }
  const int64_t slots = kCUs * resident;
  const int64_t smax = std::max<int64_t>(1, std::min(4 * slots / tiles, (K + 255) / 256));
  double best = 1e300;
  for (int64_t s = 1; s <= smax; ++s)
    best = std::min(best, (double)((tiles * s + slots - 1) / slots) / (double)s);
  for (int64_t s = 1; s <= smax; ++s)
    if ((double)((tiles * s + slots - 1) / slots) / (double)s <= best * 1.01) return s;
  return 1;
}

}  // namespace ooc
