// Memory-bound layers: ReLU, addition, SGD, softmax cross-entropy, batch
// normalisation, pooling, and the swap-integrity test op (gfx950).
//
// These kernels are bound by HBM bandwidth, not arithmetic: they stream
// with 16-byte accesses in grid-stride loops sized to fill the 256 CUs, and
// every reduction runs in a fixed order (per-slice partials written to the
// function's own variables, then summed slice by slice), so results never
// depend on scheduling or on where a variable lives.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "kernels.h"

namespace ooc {

namespace {

constexpr int TPB = 256;

unsigned grid_for(int64_t work, int64_t per_block = TPB) {
  int64_t g = (work + per_block - 1) / per_block;
  if (g < 1) g = 1;
  if (g > 16384) g = 16384;
  return (unsigned)g;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// ---------------------------------------------------------------- elementwise
template <int OP>   // 0: relu fwd, 1: relu bwd, 2: add
__global__ void ew_kernel(const float* __restrict__ a, const float* __restrict__ b,
                          float* __restrict__ y, int64_t n, bool vec) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  auto f = [](float x, float z) {
    if (OP == 0) return x > 0.f ? x : 0.f;
    if (OP == 1) return x > 0.f ? z : 0.f;
    return x + z;
  };
  int64_t done = 0;
  if (vec) {
    const int64_t n4 = n / 4;
    for (int64_t j = i; j < n4; j += stride) {
      const float4 x = reinterpret_cast<const float4*>(a)[j];
      const float4 z = OP == 0 ? x : reinterpret_cast<const float4*>(b)[j];
      reinterpret_cast<float4*>(y)[j] = make_float4(f(x.x, z.x), f(x.y, z.y), f(x.z, z.z),
                                                    f(x.w, z.w));
    }
    done = n4 * 4;
  }
  for (int64_t j = done + i; j < n; j += stride) y[j] = f(a[j], OP == 0 ? a[j] : b[j]);
}

template <int OP>
hipError_t ew(const float* a, const float* b, float* y, int64_t n, hipStream_t s) {
  const bool vec = aligned16(a) && aligned16(y) && (OP == 0 || aligned16(b));
  hipLaunchKernelGGL(ew_kernel<OP>, dim3(grid_for((n + 3) / 4)), dim3(TPB), 0, s, a, b, y, n, vec);
  return hipGetLastError();
}

// a += b in place: each element is read and written by the same lane, so the
// running gradient needs no second buffer.
__global__ void acc_kernel(float* __restrict__ a, const float* __restrict__ b, int64_t n,
                           bool vec) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t done = 0;
  if (vec) {
    const int64_t n4 = n / 4;
    for (int64_t j = i; j < n4; j += stride) {
      const float4 x = reinterpret_cast<const float4*>(a)[j];
      const float4 z = reinterpret_cast<const float4*>(b)[j];
      reinterpret_cast<float4*>(a)[j] = make_float4(x.x + z.x, x.y + z.y, x.z + z.z, x.w + z.w);
    }
    done = n4 * 4;
  }
  for (int64_t j = done + i; j < n; j += stride) a[j] = a[j] + b[j];
}

// Up to kSgdSet parameter tensors of one update function in one launch: grid row y
// updates tensor y, each element with the same arithmetic as a launch of its own.
constexpr int kSgdSet = 8;
struct SgdSet {
  float* w[kSgdSet];
  const float* g[kSgdSet];
  float* v[kSgdSet];
  int64_t n[kSgdSet];
  int32_t vec[kSgdSet];
};

__global__ void sgd_kernel(SgdSet set, float lr, float mu) {
  const int k = blockIdx.y;
  float* __restrict__ w = set.w[k];
  const float* __restrict__ g = set.g[k];
  float* __restrict__ v = set.v[k];
  const int64_t n = set.n[k];
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t done = 0;
  if (set.vec[k]) {
    const int64_t n4 = n / 4;
    for (int64_t j = i; j < n4; j += stride) {
      float4 ww = reinterpret_cast<float4*>(w)[j];
      float4 gg = reinterpret_cast<const float4*>(g)[j];
      if (v) {
        float4 vv = reinterpret_cast<float4*>(v)[j];
        vv.x = mu * vv.x + gg.x; vv.y = mu * vv.y + gg.y;
        vv.z = mu * vv.z + gg.z; vv.w = mu * vv.w + gg.w;
        reinterpret_cast<float4*>(v)[j] = vv;
        gg = vv;
      }
      ww.x -= lr * gg.x; ww.y -= lr * gg.y; ww.z -= lr * gg.z; ww.w -= lr * gg.w;
      reinterpret_cast<float4*>(w)[j] = ww;
    }
    done = n4 * 4;
  }
  for (int64_t j = done + i; j < n; j += stride) {
    float gg = g[j];
    if (v) {
      v[j] = mu * v[j] + gg;
      gg = v[j];
    }
    w[j] -= lr * gg;
  }
}

// ---------------------------------------------------------------- softmax cross-entropy
__device__ inline float wave_max(float x) {
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ inline float wave_sum(float x) {
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// one wave64 per row
__global__ void softmax_ce_rows(const float* __restrict__ z, const int32_t* __restrict__ labels,
                                float* __restrict__ loss, float* __restrict__ dz, int64_t N,
                                int64_t C) {
  const int64_t row = (int64_t)blockIdx.x * (TPB / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= N) return;
  const float* zr = z + row * C;
  float* dr = dz + row * C;
  const int32_t lab = labels[row];
  const bool ok = lab >= 0 && lab < C;
  float mx = -INFINITY;
  for (int64_t c = lane; c < C; c += 64) mx = fmaxf(mx, zr[c]);
  mx = wave_max(mx);
  float sum = 0.f;
  for (int64_t c = lane; c < C; c += 64) sum += expf(zr[c] - mx);
  sum = wave_sum(sum);
  const float inv_n = 1.f / (float)N;
  const float lse = logf(sum);
  for (int64_t c = lane; c < C; c += 64) {
    const float p = expf(zr[c] - mx - lse);
    dr[c] = ok ? (p - (c == lab ? 1.f : 0.f)) * inv_n : 0.f;
  }
  if (lane == 0) loss[row] = ok ? lse - (zr[lab] - mx) : NAN;
}

// loss[N] = mean of loss[0..N), summed in a fixed order by one workgroup of
// MEAN_T threads: float4 loads (when loss is 16-byte aligned), four of them in
// flight per thread into four accumulators, then a tree over the threads.
constexpr int MEAN_T = 1024;
__global__ __launch_bounds__(MEAN_T) void mean_rows(float* __restrict__ loss, int64_t N, bool vec) {
  __shared__ float part[MEAN_T];
  const int t = threadIdx.x;
  float a[4] = {0.f, 0.f, 0.f, 0.f};
  int64_t done = 0;
  if (vec) {
    const float4* l4 = reinterpret_cast<const float4*>(loss);
    const int64_t n4 = N / 4;
    int64_t i = t;
    for (; i + 3 * MEAN_T < n4; i += 4 * MEAN_T) {
      float4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = l4[i + u * MEAN_T];
#pragma unroll
      for (int u = 0; u < 4; ++u) a[u] += (v[u].x + v[u].y) + (v[u].z + v[u].w);
    }
    for (; i < n4; i += MEAN_T) {
      const float4 v = l4[i];
      a[0] += (v.x + v.y) + (v.z + v.w);
    }
    done = n4 * 4;
  }
  for (int64_t r = done + t; r < N; r += MEAN_T) a[1] += loss[r];
  part[t] = (a[0] + a[1]) + (a[2] + a[3]);
  __syncthreads();
  for (int w = MEAN_T / 2; w > 0; w >>= 1) {
    if (t < w) part[t] += part[t + w];
    __syncthreads();
  }
  if (t == 0) loss[N] = part[0] / (float)N;
}

// ---------------------------------------------------------------- batch normalisation
// Rows split into `slices` contiguous slices; a workgroup takes one slice and
// 64 channels: 16 channel lanes x 4 channels, 16 row lanes.
struct SliceMap {
  int64_t rows, slices, len;
  __device__ int64_t begin(int64_t s) const { return s * len; }
  __device__ int64_t end(int64_t s) const { return min(rows, (s + 1) * len); }
};

// per (slice, channel): sums of (x - shift) and (x - shift)^2, shift = x[row 0]
// (mode 0), or of dy and dy * xhat (mode 1)
template <int MODE>
__global__ void bn_partials(const float* __restrict__ x, const float* __restrict__ dy,
                            float* __restrict__ stats, SliceMap sm, int64_t C) {
  __shared__ float sa[16][64], sb[16][64];
  const int s = blockIdx.x;
  const int rl = threadIdx.x >> 4, cl = threadIdx.x & 15;
  const int64_t c0 = (int64_t)blockIdx.y * 64 + cl * 4;
  float a[4] = {0, 0, 0, 0}, b[4] = {0, 0, 0, 0};
  float sh[4] = {0, 0, 0, 0}, inv[4] = {0, 0, 0, 0};
  for (int e = 0; e < 4; ++e) {
    const int64_t c = c0 + e;
    if (c < C) {
      if (MODE == 0) {
        sh[e] = x[c];
      } else {
        sh[e] = stats[c];
        inv[e] = stats[C + c];
      }
    }
  }
  const bool vec = (C % 4 == 0) && c0 + 3 < C;
  auto add = [&](const float (&xv)[4], const float (&gv)[4]) {
    for (int e = 0; e < 4; ++e) {
      if (MODE == 0) {
        const float d = xv[e] - sh[e];
        a[e] += d;
        b[e] += d * d;
      } else {
        const float xh = (xv[e] - sh[e]) * inv[e];
        a[e] += gv[e];
        b[e] += gv[e] * xh;
      }
    }
  };
  int64_t r = sm.begin(s) + rl;
  const int64_t r_end = sm.end(s);
  if (vec) {
    // four rows' loads in flight per lane, then added in row order as below
    for (; r + 48 < r_end; r += 64) {
      float4 t[4], u[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        t[k] = *reinterpret_cast<const float4*>(&x[(r + 16 * k) * C + c0]);
        if (MODE == 1) u[k] = *reinterpret_cast<const float4*>(&dy[(r + 16 * k) * C + c0]);
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float xv[4] = {t[k].x, t[k].y, t[k].z, t[k].w};
        float gv[4] = {0, 0, 0, 0};
        if (MODE == 1) {
          gv[0] = u[k].x; gv[1] = u[k].y; gv[2] = u[k].z; gv[3] = u[k].w;
        }
        add(xv, gv);
      }
    }
  }
  for (; r < r_end; r += 16) {
    float xv[4], gv[4] = {0, 0, 0, 0};
    if (vec) {
      const float4 t = *reinterpret_cast<const float4*>(&x[r * C + c0]);
      xv[0] = t.x; xv[1] = t.y; xv[2] = t.z; xv[3] = t.w;
      if (MODE == 1) {
        const float4 u = *reinterpret_cast<const float4*>(&dy[r * C + c0]);
        gv[0] = u.x; gv[1] = u.y; gv[2] = u.z; gv[3] = u.w;
      }
    } else {
      for (int e = 0; e < 4; ++e) {
        const int64_t c = c0 + e;
        xv[e] = c < C ? x[r * C + c] : 0.f;
        if (MODE == 1) gv[e] = c < C ? dy[r * C + c] : 0.f;
      }
    }
    add(xv, gv);
  }
  for (int e = 0; e < 4; ++e) {
    sa[rl][cl * 4 + e] = a[e];
    sb[rl][cl * 4 + e] = b[e];
  }
  __syncthreads();
  if (threadIdx.x < 64) {
    const int64_t c = (int64_t)blockIdx.y * 64 + threadIdx.x;
    if (c < C) {
      float ta = 0.f, tb = 0.f;
      for (int j = 0; j < 16; ++j) {
        ta += sa[j][threadIdx.x];
        tb += sb[j][threadIdx.x];
      }
      float* part = stats + 2 * C + (int64_t)s * 2 * C;
      part[c] = ta;
      part[C + c] = tb;
    }
  }
}

// Slice partials are combined in fp64 and in a fixed order, in two passes so
// that a layer with few channels and many slices still spreads over the GPU.
// Pass 1 (more than 256 slices): workgroup (channel group, slice group g) sums its
// group's slices for 64 channels, wave w taking the slices w, w + 4, ... of
// the group in four interleaved chains, the waves added in order.  The group
// owns at least two slices; once all its waves have read them, it stores the
// two fp64 sums of each channel as bit halves in that channel's own columns of
// its first two slices, which no other workgroup reads.
__global__ __launch_bounds__(TPB) void bn_group_sums(float* __restrict__ part, int64_t C,
                                                     int64_t slices, int64_t per, int64_t groups) {
  __shared__ double sa[4][64], sb[4][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t c = (int64_t)blockIdx.x * 64 + lane;
  const int64_t g = blockIdx.y;
  const int64_t s0 = g * per, s1 = g + 1 == groups ? slices : s0 + per;
  double a[4] = {0, 0, 0, 0}, b[4] = {0, 0, 0, 0};
  if (c < C) {
    int64_t s = s0 + w;
    for (; s + 12 < s1; s += 16) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float* p = part + (s + 4 * u) * 2 * C;
        a[u] += p[c];
        b[u] += p[C + c];
      }
    }
    for (int u = 0; s < s1; s += 4, ++u) {
      const float* p = part + s * 2 * C;
      a[u] += p[c];
      b[u] += p[C + c];
    }
  }
  sa[w][lane] = (a[0] + a[1]) + (a[2] + a[3]);
  sb[w][lane] = (b[0] + b[1]) + (b[2] + b[3]);
  __syncthreads();
  if (w != 0 || c >= C) return;
  const double ta = ((sa[0][lane] + sa[1][lane]) + sa[2][lane]) + sa[3][lane];
  const double tb = ((sb[0][lane] + sb[1][lane]) + sb[2][lane]) + sb[3][lane];
  float* p0 = part + s0 * 2 * C;
  float* p1 = p0 + 2 * C;
  p0[c] = __int_as_float(__double2loint(ta));
  p0[C + c] = __int_as_float(__double2hiint(ta));
  p1[c] = __int_as_float(__double2loint(tb));
  p1[C + c] = __int_as_float(__double2hiint(tb));
}

// Pass 2 adds, per channel, either the fp64 sums of the slice groups
// (GROUPED) or the slices' float partials.  Its workgroup has 16 waves (the
// pass is a short chain of dependent loads per lane, so more waves shorten
// it); wave w takes the terms w, w + 16, ... in four interleaved chains (term
// w + 16 u + 64 i goes to chain u), the chains and then the 16 waves are added
// in order.  Forward -> mean, invstd; backward -> dgamma, dbeta.
constexpr int FIN_W = 16;
template <bool GROUPED>
__device__ inline void bn_term(const float* part, int64_t C, int64_t per, int64_t t, int64_t c,
                               double& a, double& b) {
  const float* p0 = part + t * per * 2 * C;
  if (GROUPED) {
    const float* p1 = p0 + 2 * C;
    a = __hiloint2double(__float_as_int(p0[C + c]), __float_as_int(p0[c]));
    b = __hiloint2double(__float_as_int(p1[C + c]), __float_as_int(p1[c]));
  } else {
    a = p0[c];
    b = p0[C + c];
  }
}

template <int MODE, bool GROUPED>
__global__ __launch_bounds__(64 * FIN_W) void bn_finalize(const float* __restrict__ x,
                                                          const float* __restrict__ part,
                                                          float* __restrict__ head,
                                                          float* __restrict__ dgamma,
                                                          float* __restrict__ dbeta, int64_t rows,
                                                          int64_t C, int64_t per, int64_t terms) {
  __shared__ double sa[FIN_W][64], sb[FIN_W][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t c = (int64_t)blockIdx.x * 64 + lane;
  double a[4] = {0, 0, 0, 0}, b[4] = {0, 0, 0, 0};
  if (c < C) {
    int64_t t = w;
    for (; t + 3 * FIN_W < terms; t += 4 * FIN_W) {
      double va[4], vb[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) bn_term<GROUPED>(part, C, per, t + FIN_W * u, c, va[u], vb[u]);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        a[u] += va[u];
        b[u] += vb[u];
      }
    }
    for (int u = 0; t < terms; t += FIN_W, ++u) {
      double va, vb;
      bn_term<GROUPED>(part, C, per, t, c, va, vb);
      a[u] += va;
      b[u] += vb;
    }
  }
  sa[w][lane] = (a[0] + a[1]) + (a[2] + a[3]);
  sb[w][lane] = (b[0] + b[1]) + (b[2] + b[3]);
  __syncthreads();
  if (w != 0 || c >= C) return;
  double ta = 0, tb = 0;
#pragma unroll
  for (int k = 0; k < FIN_W; ++k) {
    ta += sa[k][lane];
    tb += sb[k][lane];
  }
  if (MODE == 0) {
    const double m1 = ta / (double)rows;
    double var = tb / (double)rows - m1 * m1;
    if (var < 0) var = 0;
    head[c] = (float)((double)x[c] + m1);
    head[C + c] = (float)(1.0 / sqrt(var + 1e-5));
  } else {
    dbeta[c] = (float)ta;
    dgamma[c] = (float)tb;
  }
}

// The slice reduction over stats' partials (after the 2 C head): one pass up
// to 256 slices, else pass 1 into at most 64 groups of at least two slices
// (the last group takes the remainder) and pass 2 over the groups.
constexpr int64_t kOnePassSlices = 256;
template <int MODE>
hipError_t bn_reduce(const float* x, float* stats, float* dgamma, float* dbeta, int64_t rows,
                     int64_t C, int64_t slices, hipStream_t s) {
  const unsigned cg = (unsigned)((C + 63) / 64);
  float* part = stats + 2 * C;
  if (slices <= kOnePassSlices) {
    hipLaunchKernelGGL((bn_finalize<MODE, false>), dim3(cg), dim3(64 * FIN_W), 0, s, x, part, stats,
                       dgamma, dbeta, rows, C, (int64_t)1, slices);
    return hipGetLastError();
  }
  const int64_t groups = std::min<int64_t>(64, slices / 2), per = slices / groups;
  hipLaunchKernelGGL(bn_group_sums, dim3(cg, (unsigned)groups), dim3(TPB), 0, s, part, C, slices,
                     per, groups);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((bn_finalize<MODE, true>), dim3(cg), dim3(64 * FIN_W), 0, s, x, part, stats, dgamma,
                     dbeta, rows, C, per, groups);
  return hipGetLastError();
}

// forward: y = (x - mean) invstd gamma + beta; backward:
// dx = gamma invstd (dy - dbeta / rows - xhat dgamma / rows)
template <int MODE>
__global__ void bn_apply(const float* __restrict__ x, const float* __restrict__ dy,
                         const float* __restrict__ stats, const float* __restrict__ gamma,
                         const float* __restrict__ beta, const float* __restrict__ dgamma,
                         float* __restrict__ out, int64_t rows, int64_t C, bool vec) {
  const int64_t n = rows * C;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const float inv_rows = 1.f / (float)rows;
  auto f = [&](float xv, float gv, int64_t c) {
    const float mean = stats[c], invstd = stats[C + c];
    const float xh = (xv - mean) * invstd;
    if (MODE == 0) return xh * gamma[c] + beta[c];
    return gamma[c] * invstd * (gv - beta[c] * inv_rows - xh * dgamma[c] * inv_rows);
  };
  int64_t done = 0;
  if (vec) {
    const int64_t n4 = n / 4;
    for (int64_t j = i; j < n4; j += stride) {
      const int64_t c = (j * 4) % C;
      const float4 xv = reinterpret_cast<const float4*>(x)[j];
      float4 gv = make_float4(0, 0, 0, 0);
      if (MODE == 1) gv = reinterpret_cast<const float4*>(dy)[j];
      reinterpret_cast<float4*>(out)[j] = make_float4(f(xv.x, gv.x, c), f(xv.y, gv.y, c + 1),
                                                      f(xv.z, gv.z, c + 2), f(xv.w, gv.w, c + 3));
    }
    done = n4 * 4;
  }
  for (int64_t j = done + i; j < n; j += stride)
    out[j] = f(x[j], MODE == 1 ? dy[j] : 0.f, j % C);
}

// ---------------------------------------------------------------- pooling
__global__ void maxpool_fwd_kernel(const float* __restrict__ x, float* __restrict__ y,
                                   uint8_t* __restrict__ idx, PoolShape p) {
  const int64_t total = p.N * p.P * p.Q * p.C;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total; o += stride) {
    const int64_t c = o % p.C;
    int64_t t = o / p.C;
    const int64_t q = t % p.Q;
    t /= p.Q;
    const int64_t pp = t % p.P;
    const int64_t n = t / p.P;
    float best = 0.f;
    int bi = -1;
    for (int r = 0; r < p.k; ++r) {
      const int64_t h = pp * p.stride + r - p.pad;
      if (h < 0 || h >= p.H) continue;
      for (int s = 0; s < p.k; ++s) {
        const int64_t w = q * p.stride + s - p.pad;
        if (w < 0 || w >= p.W) continue;
        const float v = x[((n * p.H + h) * p.W + w) * p.C + c];
        if (bi < 0 || v > best) {
          best = v;
          bi = r * (int)p.k + s;
        }
      }
    }
    y[o] = best;
    idx[o] = (uint8_t)(bi < 0 ? 0 : bi);
  }
}

__global__ void maxpool_bwd_kernel(const uint8_t* __restrict__ idx, const float* __restrict__ dy,
                                   float* __restrict__ dx, PoolShape p) {
  const int64_t total = p.N * p.H * p.W * p.C;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total; o += stride) {
    const int64_t c = o % p.C;
    int64_t t = o / p.C;
    const int64_t w = t % p.W;
    t /= p.W;
    const int64_t h = t % p.H;
    const int64_t n = t / p.H;
    // output rows whose window covers h: p st - pad <= h <= p st - pad + k - 1
    int64_t plo = h + p.pad - p.k + 1;
    plo = plo <= 0 ? 0 : (plo + p.stride - 1) / p.stride;
    int64_t phi = (h + p.pad) / p.stride;
    if (phi > p.P - 1) phi = p.P - 1;
    int64_t qlo = w + p.pad - p.k + 1;
    qlo = qlo <= 0 ? 0 : (qlo + p.stride - 1) / p.stride;
    int64_t qhi = (w + p.pad) / p.stride;
    if (qhi > p.Q - 1) qhi = p.Q - 1;
    float acc = 0.f;
    for (int64_t pp = plo; pp <= phi; ++pp)
      for (int64_t q = qlo; q <= qhi; ++q) {
        const int64_t r = h - (pp * p.stride - p.pad), s = w - (q * p.stride - p.pad);
        const int64_t oi = ((n * p.P + pp) * p.Q + q) * p.C + c;
        if (idx[oi] == r * p.k + s) acc += dy[oi];
      }
    dx[o] = acc;
  }
}

// The same two pooling passes for four channels per thread (C % 4 == 0) with
// 32-bit index arithmetic (fewer than 2^31 elements): float4 data, uchar4
// indices.  Per channel the taps are visited in the same order, so results
// and ties are those of the kernels above.
struct Pool32 {
  int H, W, C4, k, st, pad, P, Q;
};
__device__ inline float comp4(const float4& v, int e) {
  return e == 0 ? v.x : e == 1 ? v.y : e == 2 ? v.z : v.w;
}

__global__ void maxpool_fwd4_kernel(const float4* __restrict__ x, float4* __restrict__ y,
                                    uchar4* __restrict__ idx, Pool32 p, int total) {
  const int stride = gridDim.x * blockDim.x;
  for (int o = blockIdx.x * blockDim.x + threadIdx.x; o < total; o += stride) {
    const int c4 = o % p.C4;
    int t = o / p.C4;
    const int q = t % p.Q;
    t /= p.Q;
    const int pp = t % p.P;
    const int n = t / p.P;
    float best[4] = {0.f, 0.f, 0.f, 0.f};
    int bi[4] = {-1, -1, -1, -1};
    for (int r = 0; r < p.k; ++r) {
      const int h = pp * p.st + r - p.pad;
      if (h < 0 || h >= p.H) continue;
      for (int s = 0; s < p.k; ++s) {
        const int w = q * p.st + s - p.pad;
        if (w < 0 || w >= p.W) continue;
        const float4 v = x[((n * p.H + h) * p.W + w) * p.C4 + c4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float ve = comp4(v, e);
          if (bi[e] < 0 || ve > best[e]) {
            best[e] = ve;
            bi[e] = r * p.k + s;
          }
        }
      }
    }
    y[o] = make_float4(best[0], best[1], best[2], best[3]);
    idx[o] = make_uchar4((unsigned char)(bi[0] < 0 ? 0 : bi[0]), (unsigned char)(bi[1] < 0 ? 0 : bi[1]),
                         (unsigned char)(bi[2] < 0 ? 0 : bi[2]), (unsigned char)(bi[3] < 0 ? 0 : bi[3]));
  }
}

__global__ void maxpool_bwd4_kernel(const uchar4* __restrict__ idx, const float4* __restrict__ dy,
                                    float4* __restrict__ dx, Pool32 p, int total) {
  const int stride = gridDim.x * blockDim.x;
  for (int o = blockIdx.x * blockDim.x + threadIdx.x; o < total; o += stride) {
    const int c4 = o % p.C4;
    int t = o / p.C4;
    const int w = t % p.W;
    t /= p.W;
    const int h = t % p.H;
    const int n = t / p.H;
    int plo = h + p.pad - p.k + 1;
    plo = plo <= 0 ? 0 : (plo + p.st - 1) / p.st;
    int phi = (h + p.pad) / p.st;
    if (phi > p.P - 1) phi = p.P - 1;
    int qlo = w + p.pad - p.k + 1;
    qlo = qlo <= 0 ? 0 : (qlo + p.st - 1) / p.st;
    int qhi = (w + p.pad) / p.st;
    if (qhi > p.Q - 1) qhi = p.Q - 1;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int pp = plo; pp <= phi; ++pp)
      for (int q = qlo; q <= qhi; ++q) {
        const int tap = (h - (pp * p.st - p.pad)) * p.k + (w - (q * p.st - p.pad));
        const int oi = ((n * p.P + pp) * p.Q + q) * p.C4 + c4;
        const uchar4 ix = idx[oi];
        const float4 g = dy[oi];
        acc[0] += ix.x == tap ? g.x : 0.f;
        acc[1] += ix.y == tap ? g.y : 0.f;
        acc[2] += ix.z == tap ? g.z : 0.f;
        acc[3] += ix.w == tap ? g.w : 0.f;
      }
    dx[o] = make_float4(acc[0], acc[1], acc[2], acc[3]);
  }
}

// workgroup of nw waves (16 for large images, 4 for small ones) per (image, 64
// channels): lane = channel, wave w sums the pixels w, w + nw, ... in four
// interleaved chains (pixel w + nw u + 4 nw i goes to chain u), so that each
// lane has four loads in flight; the chains and then the wave sums are added
// in order
constexpr int POOL_W = 16;
__global__ __launch_bounds__(64 * POOL_W) void avgpool_fwd_kernel(const float* __restrict__ x,
                                                                 float* __restrict__ y,
                                                                 int64_t HW, int64_t C) {
  __shared__ float part[POOL_W][64];
  const int nw = (int)blockDim.x >> 6;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t n = blockIdx.y;
  const int64_t c = (int64_t)blockIdx.x * 64 + lane;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  if (c < C) {
    const float* xn = x + n * HW * C + c;
    int64_t j = w;
    for (; j + 3 * nw < HW; j += 4 * nw) {
      float v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = xn[(j + nw * u) * C];
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[u] += v[u];
    }
    for (int u = 0; j < HW; j += nw, ++u) acc[u] += xn[j * C];
  }
  part[w][lane] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
  __syncthreads();
  if (w == 0 && c < C) {
    float t = 0.f;
    for (int k = 0; k < nw; ++k) t += part[k][lane];
    y[n * C + c] = t / (float)HW;
  }
}

__global__ void avgpool_bwd_kernel(const float* __restrict__ dy, float* __restrict__ dx, int64_t N,
                                   int64_t HW, int64_t C) {
  const int64_t total = N * HW * C;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const float inv = 1.f / (float)HW;
  for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total; o += stride) {
    const int64_t c = o % C, n = o / (HW * C);
    dx[o] = dy[n * C + c] * inv;
  }
}

// ---------------------------------------------------------------- test op
constexpr int kMixMax = 16;
struct MixArgs {
  const uint32_t* src[kMixMax];
  uint64_t len[kMixMax];
  int nsrc;
  uint32_t* y;
  uint64_t ylen;
  uint32_t seed;
};

__global__ void mix_kernel(MixArgs a) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t j = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; j < a.ylen; j += stride) {
    uint32_t acc = 0;
    for (int k = 0; k < a.nsrc; ++k) acc += a.src[k][j % a.len[k]];
    a.y[j] = a.seed ^ (uint32_t)(j * 2654435761ull) ^ acc;
  }
}

// ---------------------------------------------------------------- concatenation, upsampling
// One part of a channel concatenation: the rows x cp block of the part sits at
// column `off` of the rows x ct concatenation.  TO_CAT copies part -> cat,
// otherwise the concatenation's columns back into the part.  VEC moves float4
// (cp, ct and off multiples of 4).
template <bool TO_CAT, bool VEC>
__device__ inline void concat_part(const float* __restrict__ src, float* __restrict__ dst,
                                   int64_t rows, int64_t cp, int64_t ct, int64_t off) {
  const int64_t per = VEC ? cp / 4 : cp;   // units per row
  const int64_t n = rows * per;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const int64_t r = i / per, u = (i - r * per) * (VEC ? 4 : 1);
    const int64_t pi = r * cp + u, ci = r * ct + off + u;
    if (VEC) {
      if (TO_CAT)
        *reinterpret_cast<float4*>(&dst[ci]) = *reinterpret_cast<const float4*>(&src[pi]);
      else
        *reinterpret_cast<float4*>(&dst[pi]) = *reinterpret_cast<const float4*>(&src[ci]);
    } else {
      if (TO_CAT)
        dst[ci] = src[pi];
      else
        dst[pi] = src[ci];
    }
  }
}

// Up to kCatSet parts in one launch: grid row y moves part y.
constexpr int kCatSet = 16;
struct CatSet {
  float* part[kCatSet];
  int64_t cp[kCatSet], off[kCatSet];
  int32_t vec[kCatSet];
};

template <bool TO_CAT>
__global__ void concat_part_kernel(float* cat, CatSet set, int64_t rows, int64_t ct) {
  const int k = blockIdx.y;
  float* part = set.part[k];
  const float* src = TO_CAT ? part : cat;
  float* dst = TO_CAT ? cat : part;
  if (set.vec[k])
    concat_part<TO_CAT, true>(src, dst, rows, set.cp[k], ct, set.off[k]);
  else
    concat_part<TO_CAT, false>(src, dst, rows, set.cp[k], ct, set.off[k]);
}

// nearest 2x upsampling of NHWC x[N][H][W][C]: one thread per output unit
template <bool VEC>
__global__ void upsample_fwd_kernel(const float* __restrict__ x, float* __restrict__ y, int64_t N,
                                    int64_t H, int64_t W, int64_t C) {
  const int64_t per = VEC ? C / 4 : C;
  const int64_t n = N * 4 * H * W * per;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    int64_t t = i / per;
    const int64_t c = (i - t * per) * (VEC ? 4 : 1);
    const int64_t w2 = t % (2 * W);
    t /= 2 * W;
    const int64_t h2 = t % (2 * H), b = t / (2 * H);
    const int64_t src = ((b * H + h2 / 2) * W + w2 / 2) * C + c, dst = i * (VEC ? 4 : 1);
    if (VEC)
      *reinterpret_cast<float4*>(&y[dst]) = *reinterpret_cast<const float4*>(&x[src]);
    else
      y[dst] = x[src];
  }
}

// its backward: one thread per input unit, the 2 x 2 block added in a fixed order
template <bool VEC>
__global__ void upsample_bwd_kernel(const float* __restrict__ dy, float* __restrict__ dx, int64_t N,
                                    int64_t H, int64_t W, int64_t C) {
  const int64_t per = VEC ? C / 4 : C;
  const int64_t n = N * H * W * per;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    int64_t t = i / per;
    const int64_t c = (i - t * per) * (VEC ? 4 : 1);
    const int64_t w = t % W;
    t /= W;
    const int64_t h = t % H, b = t / H;
    const int64_t row = 2 * W * C;   // one output row
    const int64_t q = ((b * 2 * H + 2 * h) * 2 * W + 2 * w) * C + c;
    if (VEC) {
      const float4 a0 = *reinterpret_cast<const float4*>(&dy[q]);
      const float4 a1 = *reinterpret_cast<const float4*>(&dy[q + C]);
      const float4 a2 = *reinterpret_cast<const float4*>(&dy[q + row]);
      const float4 a3 = *reinterpret_cast<const float4*>(&dy[q + row + C]);
      *reinterpret_cast<float4*>(&dx[i * 4]) =
          make_float4(((a0.x + a1.x) + a2.x) + a3.x, ((a0.y + a1.y) + a2.y) + a3.y,
                      ((a0.z + a1.z) + a2.z) + a3.z, ((a0.w + a1.w) + a2.w) + a3.w);
    } else {
      dx[i] = ((dy[q] + dy[q + C]) + dy[q + row]) + dy[q + row + C];
    }
  }
}

}  // namespace

hipError_t relu_fwd(const float* x, float* y, int64_t n, hipStream_t s) {
  return ew<0>(x, nullptr, y, n, s);
}
hipError_t relu_bwd(const float* y, const float* dy, float* dx, int64_t n, hipStream_t s) {
  return ew<1>(y, dy, dx, n, s);
}
hipError_t add(const float* a, const float* b, float* y, int64_t n, hipStream_t s) {
  return ew<2>(a, b, y, n, s);
}

hipError_t accumulate(float* a, const float* b, int64_t n, hipStream_t s) {
  const bool vec = aligned16(a) && aligned16(b);
  hipLaunchKernelGGL(acc_kernel, dim3(grid_for((n + 3) / 4)), dim3(TPB), 0, s, a, b, n, vec);
  return hipGetLastError();
}

hipError_t sgd(int count, float* const* w, const float* const* g, float* const* v,
               const int64_t* n, float lr, float mu, hipStream_t s) {
  for (int k0 = 0; k0 < count; k0 += kSgdSet) {
    SgdSet set{};
    const int m = std::min(kSgdSet, count - k0);
    unsigned gx = 1;
    for (int k = 0; k < m; ++k) {
      set.w[k] = w[k0 + k];
      set.g[k] = g[k0 + k];
      set.v[k] = v[k0 + k];
      set.n[k] = n[k0 + k];
      set.vec[k] = aligned16(set.w[k]) && aligned16(set.g[k]) && (!set.v[k] || aligned16(set.v[k]));
      gx = std::max(gx, grid_for((set.n[k] + 3) / 4));
    }
    hipLaunchKernelGGL(sgd_kernel, dim3(gx, (unsigned)m), dim3(TPB), 0, s, set, lr, mu);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t softmax_ce(const float* logits, const int32_t* labels, float* loss, float* dlogits,
                      int64_t N, int64_t classes, hipStream_t s) {
  const int64_t rows_per_block = TPB / 64;
  hipLaunchKernelGGL(softmax_ce_rows, dim3((unsigned)((N + rows_per_block - 1) / rows_per_block)),
                     dim3(TPB), 0, s, logits, labels, loss, dlogits, N, classes);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(mean_rows, dim3(1), dim3(MEAN_T), 0, s, loss, N, aligned16(loss));
  return hipGetLastError();
}

hipError_t bn_fwd(const float* x, const float* gamma, const float* beta, float* y, float* stats,
                  int64_t rows, int64_t C, int64_t slices, hipStream_t s) {
  SliceMap sm{rows, slices, (rows + slices - 1) / slices};
  const unsigned cg = (unsigned)((C + 63) / 64);
  hipLaunchKernelGGL(bn_partials<0>, dim3((unsigned)slices, cg), dim3(TPB), 0, s, x, nullptr,
                     stats, sm, C);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if ((e = bn_reduce<0>(x, stats, nullptr, nullptr, rows, C, slices, s)) != hipSuccess) return e;
  const bool vec = C % 4 == 0 && aligned16(x) && aligned16(y);
  hipLaunchKernelGGL(bn_apply<0>, dim3(grid_for((rows * C + 3) / 4)), dim3(TPB), 0, s, x, nullptr,
                     stats, gamma, beta, nullptr, y, rows, C, vec);
  return hipGetLastError();
}

hipError_t bn_bwd(const float* x, const float* gamma, float* stats, const float* dy, float* dx,
                  float* dgamma, float* dbeta, int64_t rows, int64_t C, int64_t slices,
                  hipStream_t s) {
  SliceMap sm{rows, slices, (rows + slices - 1) / slices};
  const unsigned cg = (unsigned)((C + 63) / 64);
  hipLaunchKernelGGL(bn_partials<1>, dim3((unsigned)slices, cg), dim3(TPB), 0, s, x, dy, stats, sm,
                     C);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if ((e = bn_reduce<1>(x, stats, dgamma, dbeta, rows, C, slices, s)) != hipSuccess) return e;
  const bool vec = C % 4 == 0 && aligned16(x) && aligned16(dy) && aligned16(dx);
  // backward uses beta's slot for dbeta: dx = gamma invstd (dy - dbeta/rows - xhat dgamma/rows)
  hipLaunchKernelGGL(bn_apply<1>, dim3(grid_for((rows * C + 3) / 4)), dim3(TPB), 0, s, x, dy,
                     stats, gamma, dbeta, dgamma, dx, rows, C, vec);
  return hipGetLastError();
}

// four channels per thread with 32-bit indices when every element index fits
static bool pool_vec(const PoolShape& p, const void* a, const void* b, const void* i) {
  const int64_t big = std::max(p.N * p.H * p.W * p.C, p.N * p.P * p.Q * p.C);
  return p.C % 4 == 0 && big < (int64_t(1) << 31) && aligned16(a) && aligned16(b) &&
         ((uintptr_t)i & 3) == 0;
}
static Pool32 pool32(const PoolShape& p) {
  return Pool32{(int)p.H, (int)p.W, (int)(p.C / 4), (int)p.k, (int)p.stride, (int)p.pad, (int)p.P,
                (int)p.Q};
}

hipError_t maxpool_fwd(const float* x, float* y, uint8_t* idx, const PoolShape& p, hipStream_t s) {
  if (pool_vec(p, x, y, idx)) {
    const int total = (int)(p.N * p.P * p.Q * p.C / 4);
    hipLaunchKernelGGL(maxpool_fwd4_kernel, dim3(grid_for(total)), dim3(TPB), 0, s,
                       reinterpret_cast<const float4*>(x), reinterpret_cast<float4*>(y),
                       reinterpret_cast<uchar4*>(idx), pool32(p), total);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(maxpool_fwd_kernel, dim3(grid_for(p.N * p.P * p.Q * p.C)), dim3(TPB), 0, s, x,
                     y, idx, p);
  return hipGetLastError();
}

hipError_t maxpool_bwd(const uint8_t* idx, const float* dy, float* dx, const PoolShape& p,
                       hipStream_t s) {
  if (pool_vec(p, dy, dx, idx)) {
    const int total = (int)(p.N * p.H * p.W * p.C / 4);
    hipLaunchKernelGGL(maxpool_bwd4_kernel, dim3(grid_for(total)), dim3(TPB), 0, s,
                       reinterpret_cast<const uchar4*>(idx), reinterpret_cast<const float4*>(dy),
                       reinterpret_cast<float4*>(dx), pool32(p), total);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(maxpool_bwd_kernel, dim3(grid_for(p.N * p.H * p.W * p.C)), dim3(TPB), 0, s,
                     idx, dy, dx, p);
  return hipGetLastError();
}

hipError_t avgpool_fwd(const float* x, float* y, int64_t N, int64_t HW, int64_t C, hipStream_t s) {
  const int nw = HW >= 256 ? POOL_W : 4;
  hipLaunchKernelGGL(avgpool_fwd_kernel, dim3((unsigned)((C + 63) / 64), (unsigned)N),
                     dim3(64 * nw), 0, s, x, y, HW, C);
  return hipGetLastError();
}

hipError_t avgpool_bwd(const float* dy, float* dx, int64_t N, int64_t HW, int64_t C,
                       hipStream_t s) {
  hipLaunchKernelGGL(avgpool_bwd_kernel, dim3(grid_for(N * HW * C)), dim3(TPB), 0, s, dy, dx, N,
                     HW, C);
  return hipGetLastError();
}

// MIX: the last variable is written; the others (and the last one too when
// `y_read`) are read
hipError_t mix(void* const* ptrs, const uint64_t* words, int nvars, uint32_t seed, hipStream_t s,
               bool y_read) {
  MixArgs a{};
  int ns = 0;
  for (int j = 0; j < nvars - 1 + (y_read ? 1 : 0); ++j) {
    if (ns >= kMixMax) return hipErrorInvalidValue;
    a.src[ns] = (const uint32_t*)ptrs[j];
    a.len[ns] = words[j];
    ++ns;
  }
  a.nsrc = ns;
  a.y = (uint32_t*)ptrs[nvars - 1];
  a.ylen = words[nvars - 1];
  a.seed = seed;
  hipLaunchKernelGGL(mix_kernel, dim3(grid_for((int64_t)a.ylen)), dim3(TPB), 0, s, a);
  return hipGetLastError();
}

hipError_t concat(bool forward, float* cat, void* const* parts, const int64_t* cs, int k,
                  int64_t rows, hipStream_t s) {
  int64_t ct = 0;
  for (int j = 0; j < k; ++j) ct += cs[j];
  int64_t off = 0;
  for (int j0 = 0; j0 < k; j0 += kCatSet) {
    CatSet set{};
    const int m = std::min(kCatSet, k - j0);
    unsigned g = 1;
    for (int j = 0; j < m; ++j) {
      float* part = static_cast<float*>(parts[j0 + j]);
      const int64_t cp = cs[j0 + j];
      set.part[j] = part;
      set.cp[j] = cp;
      set.off[j] = off;
      set.vec[j] = cp % 4 == 0 && ct % 4 == 0 && off % 4 == 0 && aligned16(cat) &&
                   aligned16(part);
      g = std::max(g, grid_for(rows * (set.vec[j] ? cp / 4 : cp)));
      off += cp;
    }
    if (forward)
      hipLaunchKernelGGL(concat_part_kernel<true>, dim3(g, (unsigned)m), dim3(TPB), 0, s, cat, set,
                         rows, ct);
    else
      hipLaunchKernelGGL(concat_part_kernel<false>, dim3(g, (unsigned)m), dim3(TPB), 0, s, cat,
                         set, rows, ct);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t upsample(bool forward, const float* in, float* out, int64_t N, int64_t H, int64_t W,
                    int64_t C, hipStream_t s) {
  const bool vec = C % 4 == 0 && aligned16(in) && aligned16(out);
  const int64_t units = N * H * W * (vec ? C / 4 : C) * (forward ? 4 : 1);
  const unsigned g = grid_for(units);
  if (forward) {
    if (vec)
      hipLaunchKernelGGL(upsample_fwd_kernel<true>, dim3(g), dim3(TPB), 0, s, in, out, N, H, W, C);
    else
      hipLaunchKernelGGL(upsample_fwd_kernel<false>, dim3(g), dim3(TPB), 0, s, in, out, N, H, W, C);
  } else {
    if (vec)
      hipLaunchKernelGGL(upsample_bwd_kernel<true>, dim3(g), dim3(TPB), 0, s, in, out, N, H, W, C);
    else
      hipLaunchKernelGGL(upsample_bwd_kernel<false>, dim3(g), dim3(TPB), 0, s, in, out, N, H, W, C);
  }
  return hipGetLastError();
}

}  // namespace ooc
