// Transformer layers: embedding, LayerNorm, exact GELU and causal attention
// (gfx950).
//
// Row-wise work (LayerNorm, softmax rows) runs one wave64 per row with the
// row held in registers, lane l owning columns l, l + 64, ...; reductions
// use cross-lane shuffles, so a row's statistics are exact sums in a fixed
// order.  Column sums over rows (LayerNorm's dgamma / dbeta, the position
// embedding's gradient) go through per-slice partials summed in slice order,
// and the token embedding's gradient gathers, per vocabulary row, the
// gradient rows of the tokens carrying that id in token order.  No atomics:
// results do not depend on scheduling.
//
// Attention materialises the probabilities P = softmax(q k^T / sqrt(dh))
// per batch and head (the variable the scheduler swaps like any other):
// batched MFMA GEMMs compute q k^T into P and P v into the context, a row
// kernel applies the scale, the causal mask and the softmax in place.  The
// backward pass runs the four batched GEMMs of dv, dP, dq, dk around the row
// kernel dS = scale P (dP - rowsum(dP P)).
#include <hip/hip_runtime.h>

#include <cmath>
#include <initializer_list>

#include "kernels.h"

namespace ooc {

namespace {

constexpr int TPB = 256;

unsigned grid_for(int64_t work) {
  int64_t g = (work + TPB - 1) / TPB;
  if (g < 1) g = 1;
  if (g > 16384) g = 16384;
  return (unsigned)g;
}

__device__ inline float wave_sum(float x) {
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
__device__ inline float wave_max(float x) {
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}

// ---------------------------------------------------------------- embedding
__global__ void embed_fwd_kernel(const int32_t* __restrict__ ids, const float* __restrict__ E,
                                 const float* __restrict__ pos, float* __restrict__ y,
                                 int64_t rows, int64_t T, int64_t V, int64_t d) {
  const int64_t n = rows * d;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const int64_t r = i / d, c = i - r * d;
    const int32_t id = ids[r];
    y[i] = (id >= 0 && id < V) ? E[(int64_t)id * d + c] + pos[(r % T) * d + c] : NAN;
  }
}

// dpos[t][c] = sum over b (in order) of dy[b T + t][c]
__global__ void embed_pos_grad(const float* __restrict__ dy, float* __restrict__ dpos, int64_t B,
                               int64_t T, int64_t d) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= T * d) return;
  float acc = 0.f;
  for (int64_t b = 0; b < B; ++b) acc += dy[b * T * d + i];
  dpos[i] = acc;
}

// dE[v][c] = sum over tokens r with ids[r] == v, in token order, of dy[r][c];
// one wave per vocabulary row, 512 columns per pass
__global__ void embed_tok_grad(const int32_t* __restrict__ ids, const float* __restrict__ dy,
                               float* __restrict__ dE, int64_t N, int64_t V, int64_t d) {
  const int64_t v = (int64_t)blockIdx.x * (TPB / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (v >= V) return;
  for (int64_t c0 = 0; c0 < d; c0 += 512) {
    float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int64_t base = 0; base < N; base += 64) {
      const int64_t r = base + lane;
      const bool m = r < N && ids[r] == v;
      unsigned long long mask = __ballot(m);
      while (mask) {
        const int j = __ffsll((long long)mask) - 1;
        mask &= mask - 1;
        const float* row = dy + (base + j) * d;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int64_t c = c0 + lane + 64 * u;
          if (c < d) acc[u] += row[c];
        }
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int64_t c = c0 + lane + 64 * u;
      if (c < d) dE[v * d + c] = acc[u];
    }
  }
}

// ---------------------------------------------------------------- LayerNorm
template <int J>
__global__ __launch_bounds__(TPB) void ln_fwd_kernel(const float* __restrict__ x,
                                                     const float* __restrict__ gamma,
                                                     const float* __restrict__ beta,
                                                     float* __restrict__ y,
                                                     float* __restrict__ stats, int64_t rows,
                                                     int64_t d) {
  const int64_t r = (int64_t)blockIdx.x * (TPB / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  const float* xr = x + r * d;
  float v[J];
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int64_t c = lane + 64 * j;
    v[j] = c < d ? xr[c] : 0.f;
    s += v[j];
  }
  const float mean = wave_sum(s) / (float)d;
  float q = 0.f;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int64_t c = lane + 64 * j;
    const float t = c < d ? v[j] - mean : 0.f;
    q += t * t;
  }
  const float rstd = 1.f / sqrtf(wave_sum(q) / (float)d + 1e-5f);
  float* yr = y + r * d;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int64_t c = lane + 64 * j;
    if (c < d) yr[c] = (v[j] - mean) * rstd * gamma[c] + beta[c];
  }
  if (lane == 0) {
    stats[r] = mean;
    stats[rows + r] = rstd;
  }
}

// dx per row; per-slice partial sums of dy xhat and dy per feature, the four
// waves of the workgroup added in wave order
template <int J>
__global__ __launch_bounds__(TPB) void ln_bwd_kernel(const float* __restrict__ x,
                                                     const float* __restrict__ gamma,
                                                     const float* __restrict__ st,
                                                     const float* __restrict__ dy,
                                                     float* __restrict__ dx,
                                                     float* __restrict__ part, int64_t rows,
                                                     int64_t d, int64_t len) {
  extern __shared__ float lds[];   // [2][d]
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t s = blockIdx.x;
  const int64_t r0 = s * len, r1 = min(rows, r0 + len);
  float ag[J], ab[J], gm[J];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int64_t c = lane + 64 * j;
    ag[j] = ab[j] = 0.f;
    gm[j] = c < d ? gamma[c] : 0.f;
  }
  for (int64_t r = r0 + w; r < r1; r += TPB / 64) {
    const float mean = st[r], rstd = st[rows + r];
    float xh[J], g[J];
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int64_t c = lane + 64 * j;
      const float dv = c < d ? dy[r * d + c] : 0.f;
      xh[j] = c < d ? (x[r * d + c] - mean) * rstd : 0.f;
      g[j] = dv * gm[j];
      s1 += g[j];
      s2 += g[j] * xh[j];
      ag[j] += dv * xh[j];
      ab[j] += dv;
    }
    const float m1 = wave_sum(s1) / (float)d, m2 = wave_sum(s2) / (float)d;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int64_t c = lane + 64 * j;
      if (c < d) dx[r * d + c] = rstd * (g[j] - m1 - xh[j] * m2);
    }
  }
  for (int k = 0; k < TPB / 64; ++k) {
    if (w == k) {
#pragma unroll
      for (int j = 0; j < J; ++j) {
        const int64_t c = lane + 64 * j;
        if (c < d) {
          lds[c] = (k == 0 ? 0.f : lds[c]) + ag[j];
          lds[d + c] = (k == 0 ? 0.f : lds[d + c]) + ab[j];
        }
      }
    }
    __syncthreads();
  }
  for (int64_t c = threadIdx.x; c < 2 * d; c += TPB) part[s * 2 * d + c] = lds[c];
}

// The same two LayerNorm passes for d % 4 == 0 with 16-byte aligned rows: a lane owns the
// float4s lane, lane + 64, ... of a row.  The backward runs 8 waves per slice.
template <int J4>
__global__ __launch_bounds__(TPB) void ln_fwd4_kernel(const float4* __restrict__ x,
                                                      const float4* __restrict__ gamma,
                                                      const float4* __restrict__ beta,
                                                      float4* __restrict__ y,
                                                      float* __restrict__ stats, int64_t rows,
                                                      int64_t d) {
  const int64_t r = (int64_t)blockIdx.x * (TPB / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (r >= rows) return;
  const int64_t d4 = d / 4;
  const float4* xr = x + r * d4;
  float4 v[J4];
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < J4; ++j) {
    const int64_t c = lane + 64 * j;
    v[j] = c < d4 ? xr[c] : make_float4(0.f, 0.f, 0.f, 0.f);
    s += v[j].x + v[j].y + v[j].z + v[j].w;
  }
  const float mean = wave_sum(s) / (float)d;
  float q = 0.f;
#pragma unroll
  for (int j = 0; j < J4; ++j) {
    if (lane + 64 * j < d4) {
      const float4 t = make_float4(v[j].x - mean, v[j].y - mean, v[j].z - mean, v[j].w - mean);
      q += t.x * t.x + t.y * t.y + t.z * t.z + t.w * t.w;
    }
  }
  const float rstd = 1.f / sqrtf(wave_sum(q) / (float)d + 1e-5f);
  float4* yr = y + r * d4;
#pragma unroll
  for (int j = 0; j < J4; ++j) {
    const int64_t c = lane + 64 * j;
    if (c < d4) {
      const float4 g = gamma[c], b = beta[c];
      yr[c] = make_float4((v[j].x - mean) * rstd * g.x + b.x, (v[j].y - mean) * rstd * g.y + b.y,
                          (v[j].z - mean) * rstd * g.z + b.z, (v[j].w - mean) * rstd * g.w + b.w);
    }
  }
  if (lane == 0) {
    stats[r] = mean;
    stats[rows + r] = rstd;
  }
}

constexpr int LNB_WAVES = 8;

template <int J4>
__global__ __launch_bounds__(64 * LNB_WAVES) void ln_bwd4_kernel(
    const float4* __restrict__ x, const float4* __restrict__ gamma, const float* __restrict__ st,
    const float4* __restrict__ dy, float4* __restrict__ dx, float* __restrict__ part, int64_t rows,
    int64_t d, int64_t len) {
  extern __shared__ float4 lds4[];   // [2][d / 4]
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t s = blockIdx.x, d4 = d / 4;
  const int64_t r0 = s * len, r1 = min(rows, r0 + len);
  const float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
  float4 ag[J4], ab[J4], gm[J4];
#pragma unroll
  for (int j = 0; j < J4; ++j) {
    const int64_t c = lane + 64 * j;
    ag[j] = ab[j] = z;
    gm[j] = c < d4 ? gamma[c] : z;
  }
  for (int64_t r = r0 + w; r < r1; r += LNB_WAVES) {
    const float mean = st[r], rstd = st[rows + r];
    float4 xh[J4], g[J4];
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int j = 0; j < J4; ++j) {
      const int64_t c = lane + 64 * j;
      const float4 dv = c < d4 ? dy[r * d4 + c] : z;
      const float4 xv = c < d4 ? x[r * d4 + c] : z;
      xh[j] = c < d4 ? make_float4((xv.x - mean) * rstd, (xv.y - mean) * rstd,
                                   (xv.z - mean) * rstd, (xv.w - mean) * rstd)
                     : z;
      g[j] = make_float4(dv.x * gm[j].x, dv.y * gm[j].y, dv.z * gm[j].z, dv.w * gm[j].w);
      s1 += g[j].x + g[j].y + g[j].z + g[j].w;
      s2 += g[j].x * xh[j].x + g[j].y * xh[j].y + g[j].z * xh[j].z + g[j].w * xh[j].w;
      ag[j].x += dv.x * xh[j].x; ag[j].y += dv.y * xh[j].y;
      ag[j].z += dv.z * xh[j].z; ag[j].w += dv.w * xh[j].w;
      ab[j].x += dv.x; ab[j].y += dv.y; ab[j].z += dv.z; ab[j].w += dv.w;
    }
    const float m1 = wave_sum(s1) / (float)d, m2 = wave_sum(s2) / (float)d;
#pragma unroll
    for (int j = 0; j < J4; ++j) {
      const int64_t c = lane + 64 * j;
      if (c < d4)
        dx[r * d4 + c] = make_float4(rstd * (g[j].x - m1 - xh[j].x * m2),
                                     rstd * (g[j].y - m1 - xh[j].y * m2),
                                     rstd * (g[j].z - m1 - xh[j].z * m2),
                                     rstd * (g[j].w - m1 - xh[j].w * m2));
    }
  }
  // per-feature partials of the slice, the waves added in wave order
  for (int k = 0; k < LNB_WAVES; ++k) {
    if (w == k) {
#pragma unroll
      for (int j = 0; j < J4; ++j) {
        const int64_t c = lane + 64 * j;
        if (c < d4) {
          const float4 pa = k == 0 ? z : lds4[c], pb = k == 0 ? z : lds4[d4 + c];
          lds4[c] = make_float4(pa.x + ag[j].x, pa.y + ag[j].y, pa.z + ag[j].z, pa.w + ag[j].w);
          lds4[d4 + c] =
              make_float4(pb.x + ab[j].x, pb.y + ab[j].y, pb.z + ab[j].z, pb.w + ab[j].w);
        }
      }
    }
    __syncthreads();
  }
  const float* l = reinterpret_cast<const float*>(lds4);
  for (int64_t c = threadIdx.x; c < 2 * d; c += 64 * LNB_WAVES) part[s * 2 * d + c] = l[c];
}

// dgamma[c] / dbeta[c] = sum over slices of the partials.  A workgroup owns
// 64 features; its 16 waves take the slices s = w mod 16 in increasing order,
// and wave 0 adds the 16 results in wave order.
constexpr int FIN_WAVES = 16;
__global__ __launch_bounds__(64 * FIN_WAVES) void ln_finalize(const float* __restrict__ part,
                                                              float* __restrict__ dgamma,
                                                              float* __restrict__ dbeta, int64_t d,
                                                              int64_t slices) {
  __shared__ float sa[FIN_WAVES][64], sb[FIN_WAVES][64];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t c = (int64_t)blockIdx.x * 64 + lane;
  float a = 0.f, b = 0.f;
  if (c < d)
    for (int64_t s = w; s < slices; s += FIN_WAVES) {
      a += part[s * 2 * d + c];
      b += part[s * 2 * d + d + c];
    }
  sa[w][lane] = a;
  sb[w][lane] = b;
  __syncthreads();
  if (w == 0 && c < d) {
    float ta = 0.f, tb = 0.f;
#pragma unroll
    for (int k = 0; k < FIN_WAVES; ++k) {
      ta += sa[k][lane];
      tb += sb[k][lane];
    }
    dgamma[c] = ta;
    dbeta[c] = tb;
  }
}

// ---------------------------------------------------------------- GELU
__global__ void gelu_kernel(const float* __restrict__ x, const float* __restrict__ dy,
                            float* __restrict__ out, int64_t n, bool backward) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const float v = x[i];
    // Phi(v) through erfc: 1 + erf(v / sqrt 2) cancels to 0 in the lower tail
    const float cdf = 0.5f * erfcf(-v * 0.70710678118654752f);
    if (!backward) {
      out[i] = v * cdf;
    } else {
      const float pdf = expf(-0.5f * v * v) * 0.39894228040143268f;
      out[i] = dy[i] * (cdf + v * pdf);
    }
  }
}

// the same arithmetic four elements at a time (n % 4 == 0, 16-byte aligned pointers)
__device__ inline float gelu_at(float v, float g, bool backward) {
  const float cdf = 0.5f * erfcf(-v * 0.70710678118654752f);
  if (!backward) return v * cdf;
  const float pdf = expf(-0.5f * v * v) * 0.39894228040143268f;
  return g * (cdf + v * pdf);
}

__global__ void gelu4_kernel(const float4* __restrict__ x, const float4* __restrict__ dy,
                             float4* __restrict__ out, int64_t n4, bool backward) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    const float4 v = x[i];
    const float4 g = backward ? dy[i] : make_float4(0.f, 0.f, 0.f, 0.f);
    out[i] = make_float4(gelu_at(v.x, g.x, backward), gelu_at(v.y, g.y, backward),
                         gelu_at(v.z, g.z, backward), gelu_at(v.w, g.w, backward));
  }
}

// ---------------------------------------------------------------- attention rows
// P row (b, h, i) in place: scale, causal mask (keys j > i get 0), softmax
__global__ void attn_softmax(float* __restrict__ P, int64_t nrows, int64_t T, float scale,
                             bool causal) {
  const int64_t row = (int64_t)blockIdx.x * (TPB / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= nrows) return;
  const int64_t i = row % T;
  const int64_t n = causal ? i + 1 : T;
  float* p = P + row * T;
  float mx = -INFINITY;
  for (int64_t j = lane; j < n; j += 64) mx = fmaxf(mx, p[j] * scale);
  mx = wave_max(mx);
  float sum = 0.f;
  for (int64_t j = lane; j < n; j += 64) sum += expf(p[j] * scale - mx);
  sum = wave_sum(sum);
  const float inv = 1.f / sum;
  for (int64_t j = lane; j < T; j += 64) p[j] = j < n ? expf(p[j] * scale - mx) * inv : 0.f;
}

// The same two row operations with the row held in registers: lane l owns the float4s
// l, l + 64, ..., so a row of T <= 256 K floats (T % 4 == 0) is read once.  Under the causal
// mask, keys j >= n are not read: their P is 0, and so is their dS.
template <int K>
__global__ void attn_softmax_regs(float* __restrict__ P, int64_t nrows, int64_t T, float scale,
                                  bool causal) {
  const int64_t row = (int64_t)blockIdx.x * (TPB / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= nrows) return;
  const int64_t n = causal ? row % T + 1 : T;
  float4* p = reinterpret_cast<float4*>(P + row * T);
  float v[K][4];
  float mx = -INFINITY;
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const int64_t j0 = 4 * (lane + 64 * k);
    float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
    if (j0 < n) t = p[lane + 64 * k];
    v[k][0] = t.x; v[k][1] = t.y; v[k][2] = t.z; v[k][3] = t.w;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (j0 + e < n) mx = fmaxf(mx, v[k][e] * scale);
  }
  mx = wave_max(mx);
  float sum = 0.f;
#pragma unroll
  for (int k = 0; k < K; ++k) {
    const int64_t j0 = 4 * (lane + 64 * k);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[k][e] = j0 + e < n ? expf(v[k][e] * scale - mx) : 0.f;
      sum += v[k][e];
    }
  }
  sum = wave_sum(sum);
  const float inv = 1.f / sum;
#pragma unroll
  for (int k = 0; k < K; ++k)
    if (4 * (lane + 64 * k) < T)
      p[lane + 64 * k] = make_float4(v[k][0] * inv, v[k][1] * inv, v[k][2] * inv, v[k][3] * inv);
}

template <int K>
__global__ void attn_softmax_bwd_regs(const float* __restrict__ P, float* __restrict__ dS,
                                      int64_t nrows, int64_t T, float scale, bool causal) {
  const int64_t row = (int64_t)blockIdx.x * (TPB / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= nrows) return;
  const int64_t n = causal ? row % T + 1 : T;
  const float4* p = reinterpret_cast<const float4*>(P + row * T);
  float4* g = reinterpret_cast<float4*>(dS + row * T);
  float4 pv[K], gv[K];
  float dot = 0.f;
#pragma unroll
  for (int k = 0; k < K; ++k) {
    pv[k] = gv[k] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (4 * (lane + 64 * k) < n) {
      pv[k] = p[lane + 64 * k];
      gv[k] = g[lane + 64 * k];
    }
    dot += gv[k].x * pv[k].x + gv[k].y * pv[k].y + gv[k].z * pv[k].z + gv[k].w * pv[k].w;
  }
  dot = wave_sum(dot);
#pragma unroll
  for (int k = 0; k < K; ++k)
    if (4 * (lane + 64 * k) < T)
      g[lane + 64 * k] = make_float4(scale * pv[k].x * (gv[k].x - dot),
                                     scale * pv[k].y * (gv[k].y - dot),
                                     scale * pv[k].z * (gv[k].z - dot),
                                     scale * pv[k].w * (gv[k].w - dot));
}

// dS row in place: dS = scale P (dP - sum_j dP P).  Under the causal mask the keys
// j >= n are neither read (dP there may be unwritten) nor kept: their dS is 0.
__global__ void attn_softmax_bwd(const float* __restrict__ P, float* __restrict__ dS,
                                 int64_t nrows, int64_t T, float scale, bool causal) {
  const int64_t row = (int64_t)blockIdx.x * (TPB / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= nrows) return;
  const int64_t n = causal ? row % T + 1 : T;
  const float* p = P + row * T;
  float* g = dS + row * T;
  float dot = 0.f;
  for (int64_t j = lane; j < n; j += 64) dot += g[j] * p[j];
  dot = wave_sum(dot);
  for (int64_t j = lane; j < T; j += 64) g[j] = j < n ? scale * p[j] * (g[j] - dot) : 0.f;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

hipError_t gelu_launch(const float* x, const float* dy, float* out, int64_t n, bool backward,
                       hipStream_t s) {
  if (n % 4 == 0 && aligned16(x) && aligned16(out) && (!backward || aligned16(dy)))
    hipLaunchKernelGGL(gelu4_kernel, dim3(grid_for(n / 4)), dim3(TPB), 0, s,
                       reinterpret_cast<const float4*>(x), reinterpret_cast<const float4*>(dy),
                       reinterpret_cast<float4*>(out), n / 4, backward);
  else
    hipLaunchKernelGGL(gelu_kernel, dim3(grid_for(n)), dim3(TPB), 0, s, x, dy, out, n, backward);
  return hipGetLastError();
}

// rows of T floats: the register kernels need T % 4 == 0, T <= 1024 and an aligned base
int softmax_regs(const float* base, int64_t T) {
  if (T % 4 != 0 || T > 1024 || !aligned16(base)) return 0;
  return T <= 256 ? 1 : T <= 512 ? 2 : 4;
}

hipError_t softmax_rows(float* P, int64_t nrows, int64_t T, float scale, bool causal,
                        hipStream_t s) {
  const dim3 grid((unsigned)((nrows + 3) / 4));
  switch (softmax_regs(P, T)) {
    case 1: hipLaunchKernelGGL(attn_softmax_regs<1>, grid, dim3(TPB), 0, s, P, nrows, T, scale, causal); break;
    case 2: hipLaunchKernelGGL(attn_softmax_regs<2>, grid, dim3(TPB), 0, s, P, nrows, T, scale, causal); break;
    case 4: hipLaunchKernelGGL(attn_softmax_regs<4>, grid, dim3(TPB), 0, s, P, nrows, T, scale, causal); break;
    default: hipLaunchKernelGGL(attn_softmax, grid, dim3(TPB), 0, s, P, nrows, T, scale, causal);
  }
  return hipGetLastError();
}

hipError_t softmax_rows_bwd(const float* P, float* dS, int64_t nrows, int64_t T, float scale,
                            bool causal, hipStream_t s) {
  const dim3 grid((unsigned)((nrows + 3) / 4));
  switch (aligned16(dS) ? softmax_regs(P, T) : 0) {
    case 1: hipLaunchKernelGGL(attn_softmax_bwd_regs<1>, grid, dim3(TPB), 0, s, P, dS, nrows, T, scale, causal); break;
    case 2: hipLaunchKernelGGL(attn_softmax_bwd_regs<2>, grid, dim3(TPB), 0, s, P, dS, nrows, T, scale, causal); break;
    case 4: hipLaunchKernelGGL(attn_softmax_bwd_regs<4>, grid, dim3(TPB), 0, s, P, dS, nrows, T, scale, causal); break;
    default: hipLaunchKernelGGL(attn_softmax_bwd, grid, dim3(TPB), 0, s, P, dS, nrows, T, scale, causal);
  }
  return hipGetLastError();
}

template <int J>
hipError_t ln_fwd_j(const float* x, const float* g, const float* b, float* y, float* st,
                    int64_t rows, int64_t d, hipStream_t s) {
  hipLaunchKernelGGL(ln_fwd_kernel<J>, dim3((unsigned)((rows + 3) / 4)), dim3(TPB), 0, s, x, g, b,
                     y, st, rows, d);
  return hipGetLastError();
}

template <int J>
hipError_t ln_bwd_j(const float* x, const float* g, float* st, const float* dy, float* dx,
                    int64_t rows, int64_t d, int64_t slices, hipStream_t s) {
  const int64_t len = (rows + slices - 1) / slices;
  hipLaunchKernelGGL(ln_bwd_kernel<J>, dim3((unsigned)slices), dim3(TPB),
                     (unsigned)(2 * d * sizeof(float)), s, x, g, st, dy, dx, st + 2 * rows, rows,
                     d, len);
  return hipGetLastError();
}

}  // namespace

hipError_t embed_fwd(const int32_t* ids, const float* E, const float* pos, float* y, int64_t B,
                     int64_t T, int64_t V, int64_t d, hipStream_t s) {
  hipLaunchKernelGGL(embed_fwd_kernel, dim3(grid_for(B * T * d)), dim3(TPB), 0, s, ids, E, pos, y,
                     B * T, T, V, d);
  return hipGetLastError();
}

hipError_t embed_bwd(const int32_t* ids, const float* dy, float* dE, float* dpos, int64_t B,
                     int64_t T, int64_t V, int64_t d, hipStream_t s) {
  hipLaunchKernelGGL(embed_pos_grad, dim3((unsigned)((T * d + TPB - 1) / TPB)), dim3(TPB), 0, s,
                     dy, dpos, B, T, d);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(embed_tok_grad, dim3((unsigned)((V + 3) / 4)), dim3(TPB), 0, s, ids, dy, dE,
                     B * T, V, d);
  return hipGetLastError();
}

template <int J4>
hipError_t ln_fwd4_j(const float* x, const float* g, const float* b, float* y, float* st,
                     int64_t rows, int64_t d, hipStream_t s) {
  hipLaunchKernelGGL(ln_fwd4_kernel<J4>, dim3((unsigned)((rows + 3) / 4)), dim3(TPB), 0, s,
                     reinterpret_cast<const float4*>(x), reinterpret_cast<const float4*>(g),
                     reinterpret_cast<const float4*>(b), reinterpret_cast<float4*>(y), st, rows, d);
  return hipGetLastError();
}

template <int J4>
hipError_t ln_bwd4_j(const float* x, const float* g, float* st, const float* dy, float* dx,
                     int64_t rows, int64_t d, int64_t slices, hipStream_t s) {
  const int64_t len = (rows + slices - 1) / slices;
  hipLaunchKernelGGL(ln_bwd4_kernel<J4>, dim3((unsigned)slices), dim3(64 * LNB_WAVES),
                     (unsigned)(2 * d * sizeof(float)), s, reinterpret_cast<const float4*>(x),
                     reinterpret_cast<const float4*>(g), st, reinterpret_cast<const float4*>(dy),
                     reinterpret_cast<float4*>(dx), st + 2 * rows, rows, d, len);
  return hipGetLastError();
}

// float4 rows: d % 4 == 0, d <= dmax and every row pointer 16-byte aligned (the backward
// stops at 2048: wider rows would spill its five float4 arrays per lane)
static bool ln_vec(int64_t d, int64_t dmax, std::initializer_list<const void*> ptrs) {
  if (d % 4 != 0 || d > dmax) return false;
  for (const void* p : ptrs)
    if (!aligned16(p)) return false;
  return true;
}

#define LN4_DISPATCH(CALL)                \
  if (d <= 256) return CALL(1);           \
  if (d <= 512) return CALL(2);           \
  if (d <= 1024) return CALL(4);          \
  if (d <= 2048) return CALL(8);          \
  if (d <= 4096) return CALL(16);         \
  return hipErrorInvalidValue

#define LN_DISPATCH(CALL)                 \
  if (d <= 64) return CALL(1);            \
  if (d <= 128) return CALL(2);           \
  if (d <= 256) return CALL(4);           \
  if (d <= 512) return CALL(8);           \
  if (d <= 1024) return CALL(16);         \
  if (d <= 2048) return CALL(32);         \
  if (d <= 4096) return CALL(64);         \
  return hipErrorInvalidValue

hipError_t layernorm_fwd(const float* x, const float* gamma, const float* beta, float* y,
                         float* stats, int64_t rows, int64_t d, int64_t slices, hipStream_t s) {
  (void)slices;
  if (ln_vec(d, 4096, {x, gamma, beta, y})) {
#define LN_F4(J) ln_fwd4_j<J>(x, gamma, beta, y, stats, rows, d, s)
    LN4_DISPATCH(LN_F4);
#undef LN_F4
  }
#define LN_F(J) ln_fwd_j<J>(x, gamma, beta, y, stats, rows, d, s)
  LN_DISPATCH(LN_F);
#undef LN_F
}

hipError_t layernorm_bwd(const float* x, const float* gamma, float* stats, const float* dy,
                         float* dx, float* dgamma, float* dbeta, int64_t rows, int64_t d,
                         int64_t slices, hipStream_t s) {
  hipError_t e;
#define LN_B(J) ln_bwd_j<J>(x, gamma, stats, dy, dx, rows, d, slices, s)
#define LN_B4(J) ln_bwd4_j<J>(x, gamma, stats, dy, dx, rows, d, slices, s)
  if (ln_vec(d, 2048, {x, gamma, dy, dx}))
    e = [&]() -> hipError_t {
      if (d <= 256) return LN_B4(1);
      if (d <= 512) return LN_B4(2);
      if (d <= 1024) return LN_B4(4);
      return LN_B4(8);
    }();
  else
    e = [&]() -> hipError_t { LN_DISPATCH(LN_B); }();
#undef LN_B4
#undef LN_B
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(ln_finalize, dim3((unsigned)((d + 63) / 64)), dim3(64 * FIN_WAVES), 0, s,
                     stats + 2 * rows, dgamma, dbeta, d, slices);
  return hipGetLastError();
}


hipError_t gelu_fwd(const float* x, float* y, int64_t n, hipStream_t s) {
  return gelu_launch(x, nullptr, y, n, false, s);
}

hipError_t gelu_bwd(const float* x, const float* dy, float* dx, int64_t n, hipStream_t s) {
  return gelu_launch(x, dy, dx, n, true, s);
}

// P = softmax(q k^T / sqrt(dh)) per batch and head, masked when causal
static hipError_t attention_probs(const float* qkv, float* P, int64_t B, int64_t T, int64_t H,
                                  int64_t dh, bool causal, hipStream_t s) {
  const int64_t d = H * dh, d3 = 3 * d, TT = T * T;
  // S = q k^T into P; under the causal mask the tiles above the diagonal are left to the
  // softmax, which writes them as 0 without reading them
  BatchStrides st{H, T * d3, dh, T * d3, dh, H * TT, TT, causal ? 1 : 0};
  hipError_t e = gemm_batched(true, qkv, d3, true, qkv + d, d3, P, T, T, T, dh, B * H, st, s);
  if (e != hipSuccess) return e;
  return softmax_rows(P, B * H * T, T, 1.f / sqrtf((float)dh), causal, s);
}

hipError_t attention_fwd(const float* qkv, float* P, float* y, int64_t B, int64_t T, int64_t H,
                         int64_t dh, bool causal, hipStream_t s) {
  const int64_t d = H * dh, d3 = 3 * d, TT = T * T;
  hipError_t e = attention_probs(qkv, P, B, T, H, dh, causal, s);
  if (e != hipSuccess) return e;
  // context = P v
  BatchStrides sv{H, H * TT, TT, T * d3, dh, T * d, dh};
  return gemm_batched(true, P, T, false, qkv + 2 * d, d3, y, d, T, dh, T, B * H, sv, s);
}

// The probabilities are recomputed here rather than kept from the forward: holding them
// ([B, H, T, T], the largest activation of a layer at sequence length 512) across the step
// would make the out-of-core schedule swap them out and back in, while recomputing costs one
// q k^T product and one softmax pass.  The same kernels on the same q, k give the forward's
// P bit for bit.
hipError_t attention_bwd(const float* qkv, float* P, const float* dy, float* dqkv, float* dS,
                         int64_t B, int64_t T, int64_t H, int64_t dh, bool causal, hipStream_t s) {
  const int64_t d = H * dh, d3 = 3 * d, TT = T * T;
  hipError_t e = attention_probs(qkv, P, B, T, H, dh, causal, s);
  if (e != hipSuccess) return e;
  // dv = P^T dO
  BatchStrides s1{H, H * TT, TT, T * d, dh, T * d3, dh};
  if ((e = gemm_batched(false, P, T, false, dy, d, dqkv + 2 * d, d3, T, dh, T, B * H, s1, s)) !=
      hipSuccess)
    return e;
  // dP = dO v^T into dS (tiles above the diagonal likewise left to the softmax backward)
  BatchStrides s2{H, T * d, dh, T * d3, dh, H * TT, TT, causal ? 1 : 0};
  if ((e = gemm_batched(true, dy, d, true, qkv + 2 * d, d3, dS, T, T, T, dh, B * H, s2, s)) !=
      hipSuccess)
    return e;
  if ((e = softmax_rows_bwd(P, dS, B * H * T, T, 1.f / sqrtf((float)dh), causal, s)) !=
      hipSuccess)
    return e;
  // dq = dS k
  BatchStrides s3{H, H * TT, TT, T * d3, dh, T * d3, dh};
  if ((e = gemm_batched(true, dS, T, false, qkv + d, d3, dqkv, d3, T, dh, T, B * H, s3, s)) !=
      hipSuccess)
    return e;
  // dk = dS^T q
  return gemm_batched(false, dS, T, false, qkv, d3, dqkv + d, d3, T, dh, T, B * H, s3, s);
}

}  // namespace ooc
