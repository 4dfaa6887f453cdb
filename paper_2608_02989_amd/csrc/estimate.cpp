// Offline commitment estimator (Sec. 3.2): p_hat_d = c_d / m_d from
// verification traces, m_d counting the proposed nodes at draft position d
// (tree depth, or block offset for a chain) and c_d those on the accepted
// output prefix; and its expansion into the per-node probabilities the
// selector takes.  Counting and estimation are host-side (offline); the
// expansion runs on the device.  See include/acceptmoe.h.
#include <hip/hip_runtime.h>

#include "abi_util.hpp"
#include "acceptmoe.h"
#include "launch.hpp"

using amoe::abi::clear_err;
using amoe::abi::fail;
using amoe::abi::hip_fail;

extern "C" {

int32_t acceptmoe_commit_count(const int32_t* depth, const uint8_t* on_path, int32_t T, int32_t D, int64_t* m,
                               int64_t* c) {
  clear_err();
  if (T < 0 || D < 1) return fail(ACCEPTMOE_ERR_INVALID_ARG, "commit_count: bad sizes (T=%d D=%d)", T, D);
  if (m == nullptr || c == nullptr || (T > 0 && (depth == nullptr || on_path == nullptr)))
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "commit_count: null pointer");
  for (int t = 0; t < T; ++t) {
    const int d = depth[t];
    if (d < 0 || d >= D) continue;  // positions outside the table are not counted
    m[d] += 1;
    c[d] += on_path[t] != 0 ? 1 : 0;
  }
  return ACCEPTMOE_OK;
}

int32_t acceptmoe_commit_estimate(const int64_t* m, const int64_t* c, int32_t D, float* p_hat) {
  clear_err();
  if (D < 1) return fail(ACCEPTMOE_ERR_INVALID_ARG, "commit_estimate: D must be >= 1 (got %d)", D);
  if (m == nullptr || c == nullptr || p_hat == nullptr) return fail(ACCEPTMOE_ERR_INVALID_ARG, "commit_estimate: null pointer");
  for (int d = 0; d < D; ++d)
    if (m[d] < 0 || c[d] < 0 || c[d] > m[d])
      return fail(ACCEPTMOE_ERR_INVALID_ARG, "commit_estimate: need 0 <= c <= m at position %d", d);
  for (int d = 0; d < D; ++d)
    p_hat[d] = m[d] > 0 ? static_cast<float>(static_cast<double>(c[d]) / static_cast<double>(m[d])) : 0.0f;
  return ACCEPTMOE_OK;
}

int32_t acceptmoe_commit_expand(const float* p_hat, int32_t D, const int32_t* depth, int32_t T, float* prob,
                                void* stream) {
  clear_err();
  if (T < 0 || D < 1) return fail(ACCEPTMOE_ERR_INVALID_ARG, "commit_expand: bad sizes (T=%d D=%d)", T, D);
  if (T == 0) return ACCEPTMOE_OK;
  if (p_hat == nullptr || depth == nullptr || prob == nullptr)
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "commit_expand: null pointer");
  hipError_t e = amoe::launch_commit_expand(p_hat, D, depth, T, prob, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ACCEPTMOE_OK : hip_fail(e, "commit_expand launch");
}

}  // extern "C"
