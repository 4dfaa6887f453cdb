// C ABI of the verify-block MoE layer: host-side argument checks (before any
// HIP call), workspace sizing and kernel launches.  See include/acceptmoe.h.
#include "acceptmoe.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>

#include "abi_util.hpp"
#include "launch.hpp"

using amoe::abi::aligned;
using amoe::abi::clear_err;
using amoe::abi::fail;
using amoe::abi::hip_fail;

namespace amoe {

// Host checks of a selection call (no HIP call, no pointer dereferenced
// except the host tree_offsets); fills the kernel parameters and the tree
// offsets.  `noop` is set for an empty call (T == 0 and B == 0).
int32_t select_prepare(const char* who, const float* logits, const int32_t* parent, const int32_t* depth,
                       const float* commit_prob, const int32_t* tree_offsets, int32_t B, int32_t T, int32_t E,
                       int32_t k, double beta, int32_t mode, int32_t budget, int32_t removal_cap,
                       const uint8_t* resident_mask, uint8_t* eligible, int32_t* topk_idx, float* topk_gate,
                       int32_t* stats, SelectParams& p, TreeOffsets& offs, bool& noop) {
  noop = false;
  if (T < 0) return fail(ACCEPTMOE_ERR_INVALID_ARG, "%s: T must be >= 0 (got %d)", who, T);
  if (T == 0 && B == 0) {
    noop = true;
    return ACCEPTMOE_OK;
  }
  if (E < 1 || E > ACCEPTMOE_MAX_EXPERTS)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "%s: E must be in [1, %d] (got %d)", who, ACCEPTMOE_MAX_EXPERTS, E);
  if (k < 1 || k > E || k > ACCEPTMOE_MAX_TOPK)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "%s: k must be in [1, min(E, %d)] (got k=%d, E=%d)", who,
                ACCEPTMOE_MAX_TOPK, k, E);
  if (B < 1 || B > ACCEPTMOE_MAX_TREES)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "%s: B must be in [1, %d] (got %d)", who, ACCEPTMOE_MAX_TREES, B);
  if (!std::isfinite(beta) || beta < 0.0)
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "%s: beta must be finite and >= 0", who);
  if (mode < ACCEPTMOE_MODE_SELF_SIZING || mode > ACCEPTMOE_MODE_COUNT)
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "%s: unknown mode %d", who, mode);
  if (tree_offsets == nullptr) {
    if (B != 1) return fail(ACCEPTMOE_ERR_INVALID_ARG, "%s: tree_offsets is NULL but B = %d", who, B);
    offs.o[0] = 0;
    offs.o[1] = T;
  } else {
    if (tree_offsets[0] != 0) return fail(ACCEPTMOE_ERR_INVALID_ARG, "%s: tree_offsets[0] must be 0", who);
    for (int b = 0; b <= B; ++b) offs.o[b] = tree_offsets[b];
    for (int b = 0; b < B; ++b) {
      if (offs.o[b + 1] < offs.o[b])
        return fail(ACCEPTMOE_ERR_INVALID_ARG, "%s: tree_offsets must be non-decreasing", who);
    }
    if (offs.o[B] != T) return fail(ACCEPTMOE_ERR_INVALID_ARG, "%s: tree_offsets[B] must equal T", who);
  }
  for (int b = 0; b < B; ++b)
    if (offs.o[b + 1] - offs.o[b] > ACCEPTMOE_MAX_TREE_NODES)
      return fail(ACCEPTMOE_ERR_UNSUPPORTED, "%s: tree %d has more than %d nodes", who, b,
                  ACCEPTMOE_MAX_TREE_NODES);
  if (!eligible) return fail(ACCEPTMOE_ERR_INVALID_ARG, "%s: null eligible", who);
  if (T > 0 && (!logits || !depth || !commit_prob || !topk_idx || !topk_gate))
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "%s: null pointer", who);
  std::memset(&p, 0, sizeof p);
  p.logits = logits;
  p.parent = parent;
  p.depth = depth;
  p.prob = commit_prob;
  p.resident = resident_mask;
  p.eligible = eligible;
  p.topk_idx = topk_idx;
  p.topk_gate = topk_gate;
  p.stats = stats;
  p.beta = beta;
  p.T = T;
  p.E = E;
  p.k = k;
  p.B = B;
  p.mode = mode;
  p.budget = budget;
  p.removal_cap = removal_cap < 0 ? E : removal_cap;
  return ACCEPTMOE_OK;
}

}  // namespace amoe

extern "C" {

const char* acceptmoe_last_error(void) { return amoe::abi::g_err; }

int32_t acceptmoe_version(void) { return 303; }

// ---------------------------------------------------------------------------
size_t acceptmoe_packed_router_bytes(int32_t E, int32_t H) {
  if (E < 1 || E > ACCEPTMOE_MAX_EXPERTS || H < 16 || H % 16 != 0) return 0;
  return amoe::packed_router_bytes(E, H);
}

int32_t acceptmoe_pack_router_weights(const float* src, int32_t E, int32_t H, void* dst, void* stream) {
  clear_err();
  if (E < 1 || E > ACCEPTMOE_MAX_EXPERTS)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "pack_router: E must be in [1, %d] (got %d)", ACCEPTMOE_MAX_EXPERTS, E);
  if (H < 16 || H % 16 != 0)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "pack_router: H must be a positive multiple of 16 (got %d)", H);
  if (!src || !dst) return fail(ACCEPTMOE_ERR_INVALID_ARG, "pack_router: null pointer");
  if (!aligned(src, 16) || !aligned(dst, 16))
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "pack_router: src and dst must be 16-byte aligned");
  const char* s = reinterpret_cast<const char*>(src);
  const char* d = reinterpret_cast<const char*>(dst);
  const size_t sbytes = static_cast<size_t>(E) * H * sizeof(float), dbytes = amoe::packed_router_bytes(E, H);
  if (s < d + dbytes && d < s + sbytes) return fail(ACCEPTMOE_ERR_INVALID_ARG, "pack_router: src and dst overlap");
  hipError_t e = amoe::launch_pack_router(src, E, H, dst, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ACCEPTMOE_OK : hip_fail(e, "pack_router launch");
}

int32_t acceptmoe_route(const void* hidden, int32_t hidden_dtype, const void* router_packed, int32_t T,
                        int32_t H, int32_t E, float* logits, void* stream) {
  clear_err();
  if (T < 0) return fail(ACCEPTMOE_ERR_INVALID_ARG, "route: T must be >= 0 (got %d)", T);
  if (E < 1 || E > ACCEPTMOE_MAX_EXPERTS)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "route: E must be in [1, %d] (got %d)", ACCEPTMOE_MAX_EXPERTS, E);
  if (H < 16 || H % 16 != 0)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "route: H must be a positive multiple of 16 (got %d)", H);
  if (hidden_dtype != ACCEPTMOE_F32 && hidden_dtype != ACCEPTMOE_BF16)
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "route: unknown hidden dtype %d", hidden_dtype);
  if (T == 0) return ACCEPTMOE_OK;
  if ((T + 15) / 16 > 65535)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "route: T must be <= %d (got %d)", 65535 * 16, T);
  if (!hidden || !router_packed || !logits) return fail(ACCEPTMOE_ERR_INVALID_ARG, "route: null pointer");
  if (!aligned(hidden, 16) || !aligned(router_packed, 16) || !aligned(logits, 4))
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "route: hidden/router_packed must be 16-byte aligned");
  hipError_t e = amoe::launch_route(hidden, hidden_dtype == ACCEPTMOE_BF16, router_packed, T, H, E, logits,
                                    static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ACCEPTMOE_OK : hip_fail(e, "route launch");
}

// ---------------------------------------------------------------------------
size_t acceptmoe_select_workspace_size(int32_t T, int32_t E, int32_t k) {
  if (T < 0 || E < 1 || k < 1) return 0;
  return amoe::select_workspace_bytes(T, E, k);
}

int32_t acceptmoe_select(const float* logits, const int32_t* parent, const int32_t* depth,
                         const float* commit_prob, const int32_t* tree_offsets, int32_t B, int32_t T,
                         int32_t E, int32_t k, double beta, int32_t mode, int32_t budget,
                         int32_t removal_cap, const uint8_t* resident_mask, uint8_t* eligible,
                         int32_t* topk_idx, float* topk_gate, int32_t* stats, void* workspace,
                         size_t workspace_bytes, void* stream) {
  clear_err();
  amoe::SelectParams p;
  amoe::TreeOffsets offs;
  bool noop = false;
  const int32_t rc = amoe::select_prepare("select", logits, parent, depth, commit_prob, tree_offsets, B, T, E, k,
                                          beta, mode, budget, removal_cap, resident_mask, eligible, topk_idx,
                                          topk_gate, stats, p, offs, noop);
  if (rc != ACCEPTMOE_OK || noop) return rc;
  const size_t need = amoe::select_workspace_bytes(T, E, k);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need))
    return fail(ACCEPTMOE_ERR_WORKSPACE, "select: workspace needs %zu bytes (got %zu)", need, workspace_bytes);
  if (workspace && !aligned(workspace, 256))
    return fail(ACCEPTMOE_ERR_WORKSPACE, "select: workspace must be 256-byte aligned");
  amoe::select_carve(workspace, T, E, k, p);
  hipError_t e = amoe::launch_select(p, offs, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ACCEPTMOE_OK : hip_fail(e, "select launch");
}

// ---------------------------------------------------------------------------
static int elem_bytes(int32_t dtype) { return dtype == ACCEPTMOE_BF16 ? 2 : 4; }

size_t acceptmoe_packed_weights_bytes(int32_t dtype, int32_t E, int32_t N, int32_t K) {
  if ((dtype != ACCEPTMOE_F32 && dtype != ACCEPTMOE_BF16) || E < 1 || N < 1 || K < 1) return 0;
  return static_cast<size_t>(E) * N * K * elem_bytes(dtype);
}

int32_t acceptmoe_pack_expert_weights(const void* src, int32_t dtype, int32_t E, int32_t N, int32_t K,
                                      void* dst, void* stream) {
  clear_err();
  if (dtype != ACCEPTMOE_F32 && dtype != ACCEPTMOE_BF16)
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "pack: unknown dtype %d", dtype);
  if (E < 1 || N < 1 || K < 1) return fail(ACCEPTMOE_ERR_INVALID_ARG, "pack: E, N, K must be >= 1");
  const int kf = 64 / elem_bytes(dtype);
  if (N % 16 != 0 || K % kf != 0)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "pack: need N %% 16 == 0 and K %% %d == 0 (N=%d K=%d)", kf, N, K);
  if (!src || !dst) return fail(ACCEPTMOE_ERR_INVALID_ARG, "pack: null pointer");
  if (!aligned(src, 16) || !aligned(dst, 16))
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "pack: src and dst must be 16-byte aligned");
  const size_t bytes = static_cast<size_t>(E) * N * K * elem_bytes(dtype);
  const char* s = static_cast<const char*>(src);
  const char* d = static_cast<const char*>(dst);
  if (s < d + bytes && d < s + bytes) return fail(ACCEPTMOE_ERR_INVALID_ARG, "pack: src and dst overlap");
  hipError_t e = amoe::launch_pack(src, dtype == ACCEPTMOE_BF16, E, N, K, dst, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ACCEPTMOE_OK : hip_fail(e, "pack launch");
}

size_t acceptmoe_packed_gate_up_bytes(int32_t dtype, int32_t E, int32_t I, int32_t H) {
  if ((dtype != ACCEPTMOE_F32 && dtype != ACCEPTMOE_BF16) || E < 1 || I < 1 || H < 1) return 0;
  return amoe::packed_gate_up_bytes(dtype == ACCEPTMOE_BF16, E, I, H);
}

int32_t acceptmoe_pack_gate_up_weights(const void* w_gate, const void* w_up, int32_t dtype, int32_t E, int32_t I,
                                       int32_t H, void* dst, void* stream) {
  clear_err();
  if (dtype != ACCEPTMOE_F32 && dtype != ACCEPTMOE_BF16)
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "pack_gate_up: unknown dtype %d", dtype);
  if (E < 1 || I < 1 || H < 1) return fail(ACCEPTMOE_ERR_INVALID_ARG, "pack_gate_up: E, I, H must be >= 1");
  const int kf = 64 / elem_bytes(dtype);
  if (I % 16 != 0 || H % kf != 0)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "pack_gate_up: need I %% 16 == 0 and H %% %d == 0 (I=%d H=%d)", kf, I, H);
  if (!w_gate || !w_up || !dst) return fail(ACCEPTMOE_ERR_INVALID_ARG, "pack_gate_up: null pointer");
  if (!aligned(w_gate, 16) || !aligned(w_up, 16) || !aligned(dst, 16))
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "pack_gate_up: w_gate, w_up and dst must be 16-byte aligned");
  const size_t src_bytes = static_cast<size_t>(E) * I * H * elem_bytes(dtype);
  const size_t dst_bytes = amoe::packed_gate_up_bytes(dtype == ACCEPTMOE_BF16, E, I, H);
  const char* d = static_cast<const char*>(dst);
  for (const void* src : {w_gate, w_up}) {
    const char* s = static_cast<const char*>(src);
    if (s < d + dst_bytes && d < s + src_bytes)
      return fail(ACCEPTMOE_ERR_INVALID_ARG, "pack_gate_up: a source overlaps dst");
  }
  hipError_t e = amoe::launch_pack_gate_up(w_gate, w_up, dtype == ACCEPTMOE_BF16, E, I, H, dst,
                                           static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ACCEPTMOE_OK : hip_fail(e, "pack_gate_up launch");
}

// ---------------------------------------------------------------------------
size_t acceptmoe_moe_forward_workspace_size(int32_t T, int32_t H, int32_t I, int32_t E, int32_t k,
                                            int32_t dtype) {
  if (T < 0 || H < 1 || I < 1 || E < 1 || k < 1) return 0;
  if (dtype != ACCEPTMOE_F32 && dtype != ACCEPTMOE_BF16) return 0;
  return amoe::forward_workspace_bytes(T, H, I, E, k, dtype == ACCEPTMOE_BF16);
}

int32_t acceptmoe_moe_forward(const void* hidden, int32_t dtype, const void* w_gate_up, const void* w_down,
                              int32_t T, int32_t H, int32_t I, int32_t E, int32_t k, const int32_t* topk_idx, const float* topk_gate, float* out, void* workspace,
                              size_t workspace_bytes, void* stream) {
  clear_err();
  if (dtype != ACCEPTMOE_F32 && dtype != ACCEPTMOE_BF16)
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "forward: unknown dtype %d", dtype);
  if (T < 0) return fail(ACCEPTMOE_ERR_INVALID_ARG, "forward: T must be >= 0 (got %d)", T);
  if (E < 1 || E > ACCEPTMOE_MAX_EXPERTS)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "forward: E must be in [1, %d] (got %d)", ACCEPTMOE_MAX_EXPERTS, E);
  if (k < 1 || k > ACCEPTMOE_MAX_TOPK)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "forward: k must be in [1, %d] (got %d)", ACCEPTMOE_MAX_TOPK, k);
  const int kf = 64 / elem_bytes(dtype);
  if (H < kf || I < kf || H % kf != 0 || I % kf != 0)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "forward: H and I must be positive multiples of %d (H=%d I=%d)",
                kf, H, I);
  if (T == 0) return ACCEPTMOE_OK;
  if (static_cast<long long>(T) * k > (1ll << 30))
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "forward: T*k too large");
  if (static_cast<long long>((H / 4 + 255) / 256) * T >= (1ll << 31))
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "forward: T * ceil(H / 1024) must stay below 2^31 (T=%d H=%d)", T, H);
  if (!hidden || !w_gate_up || !w_down || !topk_idx || !topk_gate || !out)
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "forward: null pointer");
  if (!aligned(hidden, 16) || !aligned(w_gate_up, 16) || !aligned(w_down, 16) || !aligned(out, 16))
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "forward: hidden, weights and out must be 16-byte aligned");
  const size_t need = amoe::forward_workspace_bytes(T, H, I, E, k, dtype == ACCEPTMOE_BF16);
  if (workspace == nullptr || workspace_bytes < need)
    return fail(ACCEPTMOE_ERR_WORKSPACE, "forward: workspace needs %zu bytes (got %zu)", need, workspace_bytes);
  if (!aligned(workspace, 256))
    return fail(ACCEPTMOE_ERR_WORKSPACE, "forward: workspace must be 256-byte aligned");
  amoe::ForwardParams p;
  std::memset(&p, 0, sizeof p);
  p.hidden = hidden;
  p.w_gate_up = w_gate_up;
  p.w_down = w_down;
  p.topk_idx = topk_idx;
  p.topk_gate = topk_gate;
  p.out = out;
  p.T = T;
  p.H = H;
  p.I = I;
  p.E = E;
  p.k = k;
  p.is_bf16 = dtype == ACCEPTMOE_BF16;
  amoe::forward_carve(workspace, p);
  hipError_t e = amoe::launch_forward(p, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ACCEPTMOE_OK : hip_fail(e, "forward launch");
}

int32_t acceptmoe_residual_add(const void* hidden, int32_t dtype, const float* y, int32_t T, int32_t H, void* out,
                               void* stream) {
  clear_err();
  if (dtype != ACCEPTMOE_F32 && dtype != ACCEPTMOE_BF16)
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "residual_add: unknown dtype %d", dtype);
  if (T < 0 || H < 1) return fail(ACCEPTMOE_ERR_INVALID_ARG, "residual_add: bad sizes (T=%d H=%d)", T, H);
  if (H % 4 != 0) return fail(ACCEPTMOE_ERR_UNSUPPORTED, "residual_add: H must be a multiple of 4 (got %d)", H);
  if (T == 0) return ACCEPTMOE_OK;
  if (!hidden || !y || !out) return fail(ACCEPTMOE_ERR_INVALID_ARG, "residual_add: null pointer");
  if (!aligned(hidden, 16) || !aligned(y, 16) || !aligned(out, 16))
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "residual_add: pointers must be 16-byte aligned");
  hipError_t e = amoe::launch_residual_add(hidden, dtype == ACCEPTMOE_BF16, y, T, H, out, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ACCEPTMOE_OK : hip_fail(e, "residual_add launch");
}

int32_t acceptmoe_stream_read(const void* src, size_t bytes, uint32_t* sink, int32_t grid, void* stream) {
  clear_err();
  if (grid < 1 || grid > 65535) return fail(ACCEPTMOE_ERR_INVALID_ARG, "stream_read: grid must be in [1, 65535] (got %d)", grid);
  if (bytes % 16 != 0) return fail(ACCEPTMOE_ERR_INVALID_ARG, "stream_read: bytes must be a multiple of 16 (got %zu)", bytes);
  if (bytes == 0) return ACCEPTMOE_OK;
  if (!src || !sink) return fail(ACCEPTMOE_ERR_INVALID_ARG, "stream_read: null pointer");
  if (!aligned(src, 16) || !aligned(sink, 4)) return fail(ACCEPTMOE_ERR_INVALID_ARG, "stream_read: src must be 16-byte aligned");
  hipError_t e = amoe::launch_stream_read(src, bytes, sink, grid, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ACCEPTMOE_OK : hip_fail(e, "stream_read launch");
}

}  // extern "C"
