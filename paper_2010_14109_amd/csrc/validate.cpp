// Signature checks of every operation: variable count, access flags,
// attribute count and each variable's byte size against the attributes.
// A kernel indexes its buffers from the attributes alone, so nothing reaches
// the device unless these checks passed.
#include <string>

#include "internal.h"

namespace ooc {

namespace {

struct Sig {
  const char* name;
  int nvars;          // -1: variable count checked by the op's own rule
  int nattrs;         // -1: checked by the op's own rule
  uint8_t access[8];
};

const Sig kSig[OOC_OP_COUNT] = {
    {"NOOP", -1, -1, {}},
    {"LINEAR_FWD", 4, 3, {OOC_R, OOC_R, OOC_R, OOC_W}},
    {"LINEAR_BWD_W", -1, 4, {OOC_R, OOC_R, OOC_W, OOC_W}},
    {"LINEAR_BWD_X", 3, 3, {OOC_R, OOC_R, OOC_W}},
    {"RELU_FWD", 2, 1, {OOC_R, OOC_W}},
    {"RELU_BWD", 3, 1, {OOC_R, OOC_R, OOC_W}},
    {"ADD", 3, 1, {OOC_R, OOC_R, OOC_W}},
    {"SOFTMAX_CE", 4, 2, {OOC_R, OOC_R, OOC_W, OOC_W}},
    {"SGD", -1, 2, {}},
    {"CONV_FWD", 3, 11, {OOC_R, OOC_R, OOC_W}},
    {"CONV_BWD_W", -1, 12, {OOC_R, OOC_R, OOC_W, OOC_W}},
    {"CONV_BWD_X", 3, 11, {OOC_R, OOC_R, OOC_W}},
    {"BN_FWD", 5, 3, {OOC_R, OOC_R, OOC_R, OOC_W, OOC_W}},
    {"BN_BWD", 7, 3, {OOC_R, OOC_R, OOC_RW, OOC_R, OOC_W, OOC_W, OOC_W}},
    {"MAXPOOL_FWD", 3, 9, {OOC_R, OOC_W, OOC_W}},
    {"MAXPOOL_BWD", 3, 9, {OOC_R, OOC_R, OOC_W}},
    {"AVGPOOL_FWD", 2, 4, {OOC_R, OOC_W}},
    {"AVGPOOL_BWD", 2, 4, {OOC_R, OOC_W}},
    {"MIX", -1, 1, {}},
    {"EMBED_FWD", 4, 4, {OOC_R, OOC_R, OOC_R, OOC_W}},
    {"EMBED_BWD", 4, 4, {OOC_R, OOC_R, OOC_W, OOC_W}},
    {"LAYERNORM_FWD", 5, 3, {OOC_R, OOC_R, OOC_R, OOC_W, OOC_W}},
    {"LAYERNORM_BWD", 7, 3, {OOC_R, OOC_R, OOC_RW, OOC_R, OOC_W, OOC_W, OOC_W}},
    {"GELU_FWD", 2, 1, {OOC_R, OOC_W}},
    {"GELU_BWD", 3, 1, {OOC_R, OOC_R, OOC_W}},
    {"ATTENTION_FWD", 3, 5, {OOC_R, OOC_W, OOC_W}},
    {"ATTENTION_BWD", 5, 5, {OOC_R, OOC_W, OOC_R, OOC_W, OOC_W}},
    {"CONCAT_FWD", -1, -1, {}},
    {"CONCAT_BWD", -1, -1, {}},
    {"UPSAMPLE_FWD", 2, 4, {OOC_R, OOC_W}},
    {"UPSAMPLE_BWD", 2, 4, {OOC_R, OOC_W}},
    {"ACC", 2, 1, {OOC_RW, OOC_R}},
};

const int64_t kMaxElems = int64_t(1) << 40;

}  // namespace

std::string check_fn(const std::vector<Var>& vars, const Fn& fn) {
  if (fn.op < 0 || fn.op >= OOC_OP_COUNT) return "unknown operation " + std::to_string(fn.op);
  const Sig& sg = kSig[fn.op];
  const std::string nm = sg.name;
  const auto& v = fn.vars;
  const auto& a = fn.attrs;
  const int nv = (int)v.size();
  if (sg.nvars >= 0 && nv != sg.nvars)
    return nm + " takes " + std::to_string(sg.nvars) + " distinct variables, got " +
           std::to_string(nv);
  if (sg.nattrs >= 0 && (int)a.size() != sg.nattrs)
    return nm + " takes " + std::to_string(sg.nattrs) + " attributes, got " +
           std::to_string(a.size());
  if (sg.nvars >= 0)
    for (int j = 0; j < nv; ++j)
      if (v[j].access != sg.access[j])
        return nm + ": variable " + std::to_string(j) + " has the wrong access";
  for (int64_t x : a)
    if (fn.op != OOC_OP_MIX && (x < 0 || x > kMaxElems)) return nm + ": attribute out of range";
  auto B = [&](int j) { return vars[v[j].var].bytes; };
  auto need = [&](int j, int64_t bytes, const char* what) -> std::string {
    if (bytes <= 0) return nm + ": empty " + what;
    if (B(j) != (uint64_t)bytes)
      return nm + ": " + what + " has " + std::to_string(B(j)) + " bytes, attributes imply " +
             std::to_string(bytes);
    return "";
  };
  std::string e;
#define NEED(j, bytes, what) \
  if (!(e = need(j, bytes, what)).empty()) return e
  switch (fn.op) {
    case OOC_OP_NOOP:
      return "";
    case OOC_OP_LINEAR_FWD: {
      int64_t M = a[0], K = a[1], N = a[2];
      NEED(0, M * K * 4, "X");
      NEED(1, N * K * 4, "W");
      NEED(2, N * 4, "b");
      NEED(3, M * N * 4, "Y");
      return "";
    }
    case OOC_OP_LINEAR_BWD_W: {
      int64_t M = a[0], K = a[1], N = a[2], slices = a[3];
      if (slices < 1 || slices > M || slices > 65535) return nm + ": bad slice count";
      if (nv != (slices > 1 ? 5 : 4)) return nm + ": partial-sum variable iff slices > 1";
      for (int j = 0; j < nv; ++j)
        if (v[j].access != (j < 2 ? OOC_R : OOC_W)) return nm + ": wrong access";
      NEED(0, M * K * 4, "X");
      NEED(1, M * N * 4, "dY");
      NEED(2, N * K * 4, "dW");
      NEED(3, N * 4, "db");
      if (nv == 5) NEED(4, slices * (N * K + N) * 4, "partial sums");
      return "";
    }
    case OOC_OP_LINEAR_BWD_X: {
      int64_t M = a[0], K = a[1], N = a[2];
      NEED(0, N * K * 4, "W");
      NEED(1, M * N * 4, "dY");
      NEED(2, M * K * 4, "dX");
      return "";
    }
    case OOC_OP_RELU_FWD:
    case OOC_OP_RELU_BWD:
    case OOC_OP_ADD:
    case OOC_OP_ACC:
      for (int j = 0; j < nv; ++j) NEED(j, a[0] * 4, "tensor");
      return "";
    case OOC_OP_SOFTMAX_CE: {
      int64_t N = a[0], C = a[1];
      NEED(0, N * C * 4, "logits");
      NEED(1, N * 4, "labels");
      NEED(2, (N + 1) * 4, "loss");
      NEED(3, N * C * 4, "dlogits");
      return "";
    }
    case OOC_OP_SGD: {
      int64_t count = a[0], mom = a[1];
      if (count <= 0 || (mom != 0 && mom != 1)) return nm + ": bad attributes";
      const int per = mom ? 3 : 2;
      if (nv != count * per) return nm + ": variable count does not match the parameter count";
      for (int64_t p = 0; p < count; ++p) {
        const int j = (int)(p * per);
        if (v[j].access != OOC_RW || v[j + 1].access != OOC_R ||
            (mom && v[j + 2].access != OOC_RW))
          return nm + ": wrong access";
        if (B(j) % 4 || B(j + 1) != B(j) || (mom && B(j + 2) != B(j)))
          return nm + ": parameter, gradient and momentum sizes differ";
      }
      return "";
    }
    case OOC_OP_CONV_FWD:
    case OOC_OP_CONV_BWD_W:
    case OOC_OP_CONV_BWD_X: {
      int64_t N = a[0], H = a[1], W = a[2], C = a[3], K = a[4], R = a[5], S = a[6], st = a[7],
              pd = a[8], P = a[9], Q = a[10];
      if (N <= 0 || H <= 0 || W <= 0 || C <= 0 || K <= 0 || R <= 0 || S <= 0 || st <= 0)
        return nm + ": non-positive shape";
      if (pd >= R || pd >= S || H + 2 * pd < R || W + 2 * pd < S)
        return nm + ": padding or filter larger than the input allows";
      if (P != (H + 2 * pd - R) / st + 1 || Q != (W + 2 * pd - S) / st + 1)
        return nm + ": output size does not follow from the input";
      const int64_t xb = N * H * W * C * 4, wb = K * R * S * C * 4, yb = N * P * Q * K * 4;
      if (fn.op == OOC_OP_CONV_FWD) {
        NEED(0, xb, "X");
        NEED(1, wb, "W");
        NEED(2, yb, "Y");
      } else if (fn.op == OOC_OP_CONV_BWD_X) {
        NEED(0, wb, "W");
        NEED(1, yb, "dY");
        NEED(2, xb, "dX");
      } else {
        const int64_t slices = a[11];
        if (slices < 1 || slices > N * P * Q || slices > 65535) return nm + ": bad slice count";
        if (nv != (slices > 1 ? 4 : 3)) return nm + ": partial-sum variable iff slices > 1";
        if (v[0].access != OOC_R || v[1].access != OOC_R || v[2].access != OOC_W ||
            (nv == 4 && v[3].access != OOC_W))
          return nm + ": wrong access";
        NEED(0, xb, "X");
        NEED(1, yb, "dY");
        NEED(2, wb, "dW");
        if (nv == 4) NEED(3, slices * K * R * S * C * 4, "partial sums");
      }
      return "";
    }
    case OOC_OP_BN_FWD:
    case OOC_OP_BN_BWD: {
      int64_t rows = a[0], C = a[1], S = a[2];
      if (rows <= 0 || C <= 0 || S < 1 || S > rows) return nm + ": bad attributes";
      const int64_t xb = rows * C * 4, cb = C * 4, sb = (2 + 2 * S) * C * 4;
      if (fn.op == OOC_OP_BN_FWD) {
        NEED(0, xb, "X");
        NEED(1, cb, "gamma");
        NEED(2, cb, "beta");
        NEED(3, xb, "Y");
        NEED(4, sb, "stats");
      } else {
        NEED(0, xb, "X");
        NEED(1, cb, "gamma");
        NEED(2, sb, "stats");
        NEED(3, xb, "dY");
        NEED(4, xb, "dX");
        NEED(5, cb, "dgamma");
        NEED(6, cb, "dbeta");
      }
      return "";
    }
    case OOC_OP_MAXPOOL_FWD:
    case OOC_OP_MAXPOOL_BWD: {
      int64_t N = a[0], H = a[1], W = a[2], C = a[3], k = a[4], st = a[5], pd = a[6], P = a[7],
              Q = a[8];
      if (N <= 0 || H <= 0 || W <= 0 || C <= 0 || k <= 0 || k > 16 || st <= 0 || pd >= k ||
          H + 2 * pd < k || W + 2 * pd < k)
        return nm + ": bad window";
      if (P != (H + 2 * pd - k) / st + 1 || Q != (W + 2 * pd - k) / st + 1)
        return nm + ": output size does not follow from the input";
      const int64_t xb = N * H * W * C * 4, yb = N * P * Q * C * 4, ib = N * P * Q * C;
      if (fn.op == OOC_OP_MAXPOOL_FWD) {
        NEED(0, xb, "X");
        NEED(1, yb, "Y");
        NEED(2, ib, "idx");
      } else {
        NEED(0, ib, "idx");
        NEED(1, yb, "dY");
        NEED(2, xb, "dX");
      }
      return "";
    }
    case OOC_OP_AVGPOOL_FWD:
    case OOC_OP_AVGPOOL_BWD: {
      int64_t N = a[0], H = a[1], W = a[2], C = a[3];
      if (fn.op == OOC_OP_AVGPOOL_FWD) {
        NEED(0, N * H * W * C * 4, "X");
        NEED(1, N * C * 4, "Y");
      } else {
        NEED(0, N * C * 4, "dY");
        NEED(1, N * H * W * C * 4, "dX");
      }
      return "";
    }
    case OOC_OP_EMBED_FWD:
    case OOC_OP_EMBED_BWD: {
      int64_t B = a[0], T = a[1], V = a[2], d = a[3];
      if (B <= 0 || T <= 0 || V <= 0 || d <= 0 || V > INT32_MAX) return nm + ": bad attributes";
      NEED(0, B * T * 4, "ids");
      if (fn.op == OOC_OP_EMBED_FWD) {
        NEED(1, V * d * 4, "E");
        NEED(2, T * d * 4, "pos");
        NEED(3, B * T * d * 4, "Y");
      } else {
        NEED(1, B * T * d * 4, "dY");
        NEED(2, V * d * 4, "dE");
        NEED(3, T * d * 4, "dpos");
      }
      return "";
    }
    case OOC_OP_LAYERNORM_FWD:
    case OOC_OP_LAYERNORM_BWD: {
      int64_t rows = a[0], d = a[1], S = a[2];
      if (rows <= 0 || d <= 0 || d > 4096 || S < 1 || S > rows) return nm + ": bad attributes";
      const int64_t xb = rows * d * 4, cb = d * 4, sb = (2 * rows + 2 * S * d) * 4;
      if (fn.op == OOC_OP_LAYERNORM_FWD) {
        NEED(0, xb, "X");
        NEED(1, cb, "gamma");
        NEED(2, cb, "beta");
        NEED(3, xb, "Y");
        NEED(4, sb, "stats");
      } else {
        NEED(0, xb, "X");
        NEED(1, cb, "gamma");
        NEED(2, sb, "stats");
        NEED(3, xb, "dY");
        NEED(4, xb, "dX");
        NEED(5, cb, "dgamma");
        NEED(6, cb, "dbeta");
      }
      return "";
    }
    case OOC_OP_GELU_FWD:
    case OOC_OP_GELU_BWD:
      for (int j = 0; j < nv; ++j) NEED(j, a[0] * 4, "tensor");
      return "";
    case OOC_OP_ATTENTION_FWD:
    case OOC_OP_ATTENTION_BWD: {
      int64_t B = a[0], T = a[1], H = a[2], dh = a[3], causal = a[4];
      if (B <= 0 || T <= 0 || H <= 0 || dh <= 0 || (causal != 0 && causal != 1) ||
          B * H > 65535)
        return nm + ": bad attributes";
      const int64_t qb = B * T * 3 * H * dh * 4, pb = B * H * T * T * 4, yb = B * T * H * dh * 4;
      NEED(0, qb, "qkv");
      if (fn.op == OOC_OP_ATTENTION_FWD) {
        NEED(1, pb, "P");
        NEED(2, yb, "Y");
      } else {
        NEED(1, pb, "P");
        NEED(2, yb, "dY");
        NEED(3, qb, "dqkv");
        NEED(4, pb, "dS");
      }
      return "";
    }
    case OOC_OP_CONCAT_FWD:
    case OOC_OP_CONCAT_BWD: {
      const int k = nv - 1;
      if (k < 1 || k > 64 || (int)a.size() != 1 + k)
        return nm + ": takes 1 + k variables and 1 + k attributes, k <= 64";
      const bool fwd = fn.op == OOC_OP_CONCAT_FWD;
      const int out = fwd ? k : 0;   // the concatenated tensor
      for (int j = 0; j < nv; ++j) {
        const uint8_t want = fwd ? (j == k ? OOC_W : OOC_R) : (j == 0 ? OOC_R : OOC_W);
        if (v[j].access != want) return nm + ": wrong access";
      }
      const int64_t rows = a[0];
      int64_t total = 0;
      for (int j = 1; j <= k; ++j) {
        if (a[j] <= 0) return nm + ": non-positive channel count";
        total += a[j];
      }
      if (rows <= 0 || rows * total > kMaxElems) return nm + ": bad attributes";
      for (int j = 0; j < k; ++j) NEED(fwd ? j : j + 1, rows * a[1 + j] * 4, "part");
      NEED(out, rows * total * 4, "concatenation");
      return "";
    }
    case OOC_OP_UPSAMPLE_FWD:
    case OOC_OP_UPSAMPLE_BWD: {
      const int64_t N = a[0], H = a[1], W = a[2], C = a[3];
      if (N <= 0 || H <= 0 || W <= 0 || C <= 0) return nm + ": non-positive shape";
      const int64_t small = N * H * W * C * 4, big = 4 * small;
      NEED(0, fn.op == OOC_OP_UPSAMPLE_FWD ? small : big, "input");
      NEED(1, fn.op == OOC_OP_UPSAMPLE_FWD ? big : small, "output");
      return "";
    }
    case OOC_OP_MIX: {
      if (nv < 1 || nv > 16) return nm + ": takes 1 to 16 variables";
      for (int j = 0; j < nv; ++j) {
        if (B(j) % 4) return nm + ": sizes must be multiples of 4";
        const bool last = j == nv - 1;
        if (!last && v[j].access != OOC_R) return nm + ": only the last variable is written";
        if (last && !(v[j].access & OOC_W)) return nm + ": the last variable must be written";
      }
      return "";
    }
  }
#undef NEED
  return "unknown operation";
}

}  // namespace ooc
