// Host half of the suffix QKV projection: the rotary-embedding angle table.
//
// With a reused prefix of P tokens, the layer work left for a request is its S
// suffix tokens (paper Sec. 1 and 2.1), and it starts with projecting each
// suffix token to its query, key and value heads; queries and keys are then
// rotated by the rotary position embedding of their absolute position P + i
// (the decoder-only model family the paper measures, Sec. 4). The table holds
// cos and sin of p * theta_j, theta_j = base^(-2j/D), evaluated in double
// precision and rounded once to fp32, so the kernel needs no transcendental
// function and its result does not depend on a device math library.

#include <cmath>
#include <cstdint>
#include <string>

#include "cw_internal.h"

extern "C" cw_status cw_rope_table(int32_t n_positions, int32_t head_dim, double base, float* out) {
  if (n_positions < 0) return cw::fail(CW_EINVAL, "n_positions must be >= 0");
  if (head_dim < 2 || head_dim % 2 != 0 || head_dim > 1024)
    return cw::fail(CW_EINVAL, "head_dim must be even and in [2, 1024]");
  if (!(base > 1.0) || !std::isfinite(base)) return cw::fail(CW_EINVAL, "base must be finite and > 1");
  if (!out && n_positions > 0) return cw::fail(CW_EINVAL, "out is NULL");
  const int32_t half = head_dim / 2;
  for (int32_t j = 0; j < half; ++j) {
    const double theta = std::pow(base, -2.0 * double(j) / double(head_dim));
    for (int32_t p = 0; p < n_positions; ++p) {
      const double a = double(p) * theta;
      float* e = out + (int64_t(p) * half + j) * 2;
      e[0] = float(std::cos(a));
      e[1] = float(std::sin(a));
    }
  }
  return cw::ok();
}
