// Maps a registered function to its kernel launches.  Shapes come from the
// attributes, which ooc_add_fn has checked against every variable's size.
#include <algorithm>

#include "kernels.h"

namespace ooc {

hipError_t launch_fn(const Fn& fn, void* const* p, const uint64_t* bytes, float lr, float mu,
                     hipStream_t s) {
  const auto& a = fn.attrs;
  auto F = [&](int j) { return static_cast<float*>(p[j]); };
  auto conv = [&]() {
    return ConvShape{a[0], a[1], a[2], a[3], a[4], a[5], a[6], a[7], a[8], a[9], a[10]};
  };
  auto pool = [&]() { return PoolShape{a[0], a[1], a[2], a[3], a[4], a[5], a[6], a[7], a[8]}; };
  switch (fn.op) {
    case OOC_OP_NOOP:
      return hipSuccess;
    case OOC_OP_LINEAR_FWD:
      return linear_fwd(F(0), F(1), F(2), F(3), a[0], a[1], a[2], s);
    case OOC_OP_LINEAR_BWD_W:
      return linear_bwd_w(F(0), F(1), F(2), F(3), a[3] > 1 ? F(4) : nullptr, a[3], a[0], a[1], a[2],
                          s);
    case OOC_OP_LINEAR_BWD_X:
      return linear_bwd_x(F(0), F(1), F(2), a[0], a[1], a[2], s);
    case OOC_OP_RELU_FWD:
      return relu_fwd(F(0), F(1), a[0], s);
    case OOC_OP_RELU_BWD:
      return relu_bwd(F(0), F(1), F(2), a[0], s);
    case OOC_OP_ADD:
      return add(F(0), F(1), F(2), a[0], s);
    case OOC_OP_ACC:
      return accumulate(F(0), F(1), a[0], s);
    case OOC_OP_SOFTMAX_CE:
      return softmax_ce(F(0), static_cast<const int32_t*>(p[1]), F(2), F(3), a[0], a[1], s);
    case OOC_OP_SGD: {
      const int per = a[1] ? 3 : 2;
      float* w[64];
      const float* g[64];
      float* v[64];
      int64_t n[64];
      for (int64_t k0 = 0; k0 < a[0]; k0 += 64) {
        const int m = (int)std::min<int64_t>(64, a[0] - k0);
        for (int k = 0; k < m; ++k) {
          const int j = (int)((k0 + k) * per);
          w[k] = F(j);
          g[k] = F(j + 1);
          v[k] = a[1] ? F(j + 2) : nullptr;
          n[k] = (int64_t)(bytes[j] / 4);
        }
        hipError_t e = sgd(m, w, g, v, n, lr, mu, s);
        if (e != hipSuccess) return e;
      }
      return hipSuccess;
    }
    case OOC_OP_MIX: {
      const int n = (int)fn.vars.size();
      uint64_t words[64];
      if (n > 64) return hipErrorInvalidValue;
      for (int j = 0; j < n; ++j) words[j] = bytes[j] / 4;
      return mix(p, words, n, (uint32_t)a[0], s, (fn.vars[n - 1].access & OOC_R) != 0);
    }
    case OOC_OP_CONV_FWD:
      return conv_fwd(F(0), F(1), F(2), conv(), s);
    case OOC_OP_CONV_BWD_X:
      return conv_bwd_x(F(0), F(1), F(2), conv(), s);
    case OOC_OP_CONV_BWD_W:
      return conv_bwd_w(F(0), F(1), F(2), a[11] > 1 ? F(3) : nullptr, a[11], conv(), s);
    case OOC_OP_BN_FWD:
      return bn_fwd(F(0), F(1), F(2), F(3), F(4), a[0], a[1], a[2], s);
    case OOC_OP_BN_BWD:
      return bn_bwd(F(0), F(1), F(2), F(3), F(4), F(5), F(6), a[0], a[1], a[2], s);
    case OOC_OP_MAXPOOL_FWD:
      return maxpool_fwd(F(0), F(1), static_cast<uint8_t*>(p[2]), pool(), s);
    case OOC_OP_MAXPOOL_BWD:
      return maxpool_bwd(static_cast<const uint8_t*>(p[0]), F(1), F(2), pool(), s);
    case OOC_OP_AVGPOOL_FWD:
      return avgpool_fwd(F(0), F(1), a[0], a[1] * a[2], a[3], s);
    case OOC_OP_AVGPOOL_BWD:
      return avgpool_bwd(F(0), F(1), a[0], a[1] * a[2], a[3], s);
    case OOC_OP_EMBED_FWD:
      return embed_fwd(static_cast<const int32_t*>(p[0]), F(1), F(2), F(3), a[0], a[1], a[2],
                       a[3], s);
    case OOC_OP_EMBED_BWD:
      return embed_bwd(static_cast<const int32_t*>(p[0]), F(1), F(2), F(3), a[0], a[1], a[2],
                       a[3], s);
    case OOC_OP_LAYERNORM_FWD:
      return layernorm_fwd(F(0), F(1), F(2), F(3), F(4), a[0], a[1], a[2], s);
    case OOC_OP_LAYERNORM_BWD:
      return layernorm_bwd(F(0), F(1), F(2), F(3), F(4), F(5), F(6), a[0], a[1], a[2], s);
    case OOC_OP_GELU_FWD:
      return gelu_fwd(F(0), F(1), a[0], s);
    case OOC_OP_GELU_BWD:
      return gelu_bwd(F(0), F(1), F(2), a[0], s);
    case OOC_OP_ATTENTION_FWD:
      return attention_fwd(F(0), F(1), F(2), a[0], a[1], a[2], a[3], a[4] != 0, s);
    case OOC_OP_ATTENTION_BWD:
      return attention_bwd(F(0), F(1), F(2), F(3), F(4), a[0], a[1], a[2], a[3], a[4] != 0, s);
    case OOC_OP_CONCAT_FWD: {
      const int k = (int)fn.vars.size() - 1;
      return concat(true, F(k), p, a.data() + 1, k, a[0], s);
    }
    case OOC_OP_CONCAT_BWD: {
      const int k = (int)fn.vars.size() - 1;
      return concat(false, F(0), p + 1, a.data() + 1, k, a[0], s);
    }
    case OOC_OP_UPSAMPLE_FWD:
      return upsample(true, F(0), F(1), a[0], a[1], a[2], a[3], s);
    case OOC_OP_UPSAMPLE_BWD:
      return upsample(false, F(0), F(1), a[0], a[1], a[2], a[3], s);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace ooc
