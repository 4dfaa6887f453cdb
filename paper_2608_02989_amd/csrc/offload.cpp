// Physical expert offload (Sec. 3.4, offload paragraph; Sec. 4, offload
// setup): a per-layer pool of X expert slots in HBM, the full packed expert
// stacks in pinned host memory, least-recently-used residency, synchronous
// on-demand host-to-device loads, and token waves when a block's routed union
// does not fit in the pool.  Host-side runtime state and bookkeeping; the
// copies are stream-ordered hipMemcpyAsync calls, so the forward launched
// after a wave on the same stream sees its experts.  See include/acceptmoe.h.
#include <hip/hip_runtime.h>

#include <cstring>
#include <vector>

#include "abi_util.hpp"
#include "acceptmoe.h"
#include "launch.hpp"

using amoe::abi::aligned;
using amoe::abi::clear_err;
using amoe::abi::fail;
using amoe::abi::hip_fail;

namespace {

constexpr uint32_t kPoolMagic = 0x4c4f4f50u;  // "POOL"

// Caller-owned host block: header, then expert_in[X], stamp[X], slot_of[E].
struct PoolHeader {
  uint32_t magic;
  int32_t X, E;
  int32_t pad;
  int64_t clock;  // waves served so far (recency time)
};

struct PoolView {
  PoolHeader* h;
  int32_t* expert_in;  // slot -> expert, -1 empty
  int64_t* stamp;      // slot -> wave time of the last use, -1 never used
  int32_t* slot_of;    // expert -> slot, -1 not resident
};

size_t pool_bytes(int X, int E) {
  return sizeof(PoolHeader) + sizeof(int64_t) * X + sizeof(int32_t) * (static_cast<size_t>(X) + E);
}

PoolView view(void* state) {
  PoolView v;
  char* c = static_cast<char*>(state);
  v.h = reinterpret_cast<PoolHeader*>(c);
  c += sizeof(PoolHeader);
  v.stamp = reinterpret_cast<int64_t*>(c);
  c += sizeof(int64_t) * v.h->X;
  v.expert_in = reinterpret_cast<int32_t*>(c);
  c += sizeof(int32_t) * v.h->X;
  v.slot_of = reinterpret_cast<int32_t*>(c);
  return v;
}

bool pool_ok(const void* state) {
  if (state == nullptr || !aligned(state, 8)) return false;
  const PoolHeader* h = static_cast<const PoolHeader*>(state);
  return h->magic == kPoolMagic && h->X >= 1 && h->E >= 1 && h->E <= ACCEPTMOE_MAX_EXPERTS;
}

// distinct experts in [0, E) of routing row `row` (k entries), first
// occurrence kept; returns how many
int row_experts(const int32_t* row, int k, int E, int32_t* out) {
  int n = 0;
  for (int j = 0; j < k; ++j) {
    const int e = row[j];
    if (e < 0 || e >= E) continue;
    bool dup = false;
    for (int q = 0; q < n; ++q) dup = dup || out[q] == e;
    if (!dup) out[n++] = e;
  }
  return n;
}

}  // namespace

extern "C" {

size_t acceptmoe_pool_state_bytes(int32_t X, int32_t E) {
  if (X < 1 || E < 1 || E > ACCEPTMOE_MAX_EXPERTS) return 0;
  return pool_bytes(X, E);
}

int32_t acceptmoe_pool_init(void* state, size_t state_bytes, int32_t X, int32_t E) {
  clear_err();
  if (X < 1 || E < 1 || E > ACCEPTMOE_MAX_EXPERTS)
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "pool_init: need X >= 1 and 1 <= E <= %d (X=%d E=%d)",
                ACCEPTMOE_MAX_EXPERTS, X, E);
  if (state == nullptr || !aligned(state, 8)) return fail(ACCEPTMOE_ERR_INVALID_ARG, "pool_init: state must be 8-byte aligned host memory");
  if (state_bytes < pool_bytes(X, E))
    return fail(ACCEPTMOE_ERR_WORKSPACE, "pool_init: state needs %zu bytes (got %zu)", pool_bytes(X, E), state_bytes);
  PoolHeader* h = static_cast<PoolHeader*>(state);
  h->magic = kPoolMagic;
  h->X = X;
  h->E = E;
  h->pad = 0;
  h->clock = 0;
  PoolView v = view(state);
  for (int s = 0; s < X; ++s) {
    v.expert_in[s] = -1;
    v.stamp[s] = -1;
  }
  for (int e = 0; e < E; ++e) v.slot_of[e] = -1;
  return ACCEPTMOE_OK;
}

int32_t acceptmoe_pool_resident_mask(const void* state, uint8_t* mask) {
  clear_err();
  if (!pool_ok(state)) return fail(ACCEPTMOE_ERR_INVALID_ARG, "pool_resident_mask: not an initialised pool state");
  if (mask == nullptr) return fail(ACCEPTMOE_ERR_INVALID_ARG, "pool_resident_mask: null mask");
  PoolView v = view(const_cast<void*>(state));
  for (int e = 0; e < v.h->E; ++e) mask[e] = v.slot_of[e] >= 0 ? 1 : 0;
  return ACCEPTMOE_OK;
}

int32_t acceptmoe_pool_plan_waves(const int32_t* topk_idx, int32_t T, int32_t k, int32_t E, int32_t X,
                                  int32_t* wave_of, int32_t* n_waves) {
  clear_err();
  if (T < 0 || k < 1 || k > ACCEPTMOE_MAX_TOPK || E < 1 || E > ACCEPTMOE_MAX_EXPERTS || X < 1)
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "pool_plan_waves: bad sizes (T=%d k=%d E=%d X=%d)", T, k, E, X);
  if (n_waves == nullptr || (T > 0 && (topk_idx == nullptr || wave_of == nullptr)))
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "pool_plan_waves: null pointer");
  std::vector<uint8_t> in_wave(E, 0);
  int32_t mine[ACCEPTMOE_MAX_TOPK];
  int w = 0, union_size = 0;
  for (int t = 0; t < T; ++t) {
    const int n = row_experts(topk_idx + static_cast<size_t>(t) * k, k, E, mine);
    if (n > X) return fail(ACCEPTMOE_ERR_UNSUPPORTED, "pool_plan_waves: token %d routes to %d experts > X = %d", t, n, X);
    int fresh = 0;
    for (int q = 0; q < n; ++q) fresh += in_wave[mine[q]] ? 0 : 1;
    if (union_size > 0 && union_size + fresh > X) {  // start the next wave with this token
      ++w;
      std::fill(in_wave.begin(), in_wave.end(), 0);
      union_size = 0;
      fresh = n;
    }
    for (int q = 0; q < n; ++q) in_wave[mine[q]] = 1;
    union_size += fresh;
    wave_of[t] = w;
  }
  *n_waves = T > 0 ? w + 1 : 0;
  return ACCEPTMOE_OK;
}

int32_t acceptmoe_pool_serve_wave(void* state, const int32_t* topk_idx, const int32_t* wave_of, int32_t wave,
                                  int32_t T, int32_t k, const void* host_gate_up, const void* host_down,
                                  void* pool_gate_up, void* pool_down, size_t gate_up_bytes, size_t down_bytes,
                                  int32_t* slot_idx, int64_t* stats, void* stream) {
  clear_err();
  if (!pool_ok(state)) return fail(ACCEPTMOE_ERR_INVALID_ARG, "pool_serve_wave: not an initialised pool state");
  if (T < 0 || k < 1 || k > ACCEPTMOE_MAX_TOPK || wave < 0)
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "pool_serve_wave: bad sizes (T=%d k=%d wave=%d)", T, k, wave);
  if (stats == nullptr || (T > 0 && (topk_idx == nullptr || wave_of == nullptr || slot_idx == nullptr)))
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "pool_serve_wave: null pointer");
  const bool copy = pool_gate_up != nullptr;
  if (copy && (host_gate_up == nullptr || host_down == nullptr || pool_down == nullptr))
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "pool_serve_wave: give all four weight pointers, or none (bookkeeping only)");
  if (copy && (gate_up_bytes == 0 || down_bytes == 0))
    return fail(ACCEPTMOE_ERR_INVALID_ARG, "pool_serve_wave: per-expert byte counts must be positive");
  PoolView v = view(state);
  const int X = v.h->X, E = v.h->E;
  // the wave's routed union
  std::vector<uint8_t> needed(E, 0);
  int32_t mine[ACCEPTMOE_MAX_TOPK];
  int n_needed = 0;
  for (int t = 0; t < T; ++t) {
    if (wave_of[t] != wave) continue;
    const int n = row_experts(topk_idx + static_cast<size_t>(t) * k, k, E, mine);
    for (int q = 0; q < n; ++q) {
      n_needed += needed[mine[q]] ? 0 : 1;
      needed[mine[q]] = 1;
    }
  }
  if (n_needed > X) return fail(ACCEPTMOE_ERR_UNSUPPORTED, "pool_serve_wave: wave %d routes to %d experts > X = %d", wave, n_needed, X);
  const int64_t now = ++v.h->clock;
  const size_t per_expert = gate_up_bytes + down_bytes;
  hipStream_t st = static_cast<hipStream_t>(stream);
  for (int e = 0; e < E; ++e) {
    if (!needed[e]) continue;
    ++stats[ACCEPTMOE_POOL_ACCESSES];
    int s = v.slot_of[e];
    if (s >= 0) {
      ++stats[ACCEPTMOE_POOL_HITS];
    } else {
      // victim: the oldest slot whose expert this wave does not use (empty
      // slots are the oldest), lower slot index on equal stamps
      int best = -1;
      for (int j = 0; j < X; ++j) {
        const int held = v.expert_in[j];
        if (held >= 0 && needed[held]) continue;
        if (best < 0 || v.stamp[j] < v.stamp[best]) best = j;
      }
      if (best < 0)  // cannot happen while the wave's union fits in X slots (checked above)
        return fail(ACCEPTMOE_ERR_INVALID_ARG, "pool_serve_wave: no slot to evict for expert %d", e);
      s = best;
      if (v.expert_in[s] >= 0) v.slot_of[v.expert_in[s]] = -1;
      v.expert_in[s] = e;
      v.slot_of[e] = s;
      ++stats[ACCEPTMOE_POOL_MISSES];
      stats[ACCEPTMOE_POOL_H2D_BYTES] += static_cast<int64_t>(per_expert);
      if (copy) {
        hipError_t err = hipMemcpyAsync(static_cast<char*>(pool_gate_up) + s * gate_up_bytes,
                                        static_cast<const char*>(host_gate_up) + e * gate_up_bytes, gate_up_bytes,
                                        hipMemcpyHostToDevice, st);
        if (err == hipSuccess)
          err = hipMemcpyAsync(static_cast<char*>(pool_down) + s * down_bytes,
                               static_cast<const char*>(host_down) + e * down_bytes, down_bytes,
                               hipMemcpyHostToDevice, st);
        if (err != hipSuccess) return hip_fail(err, "pool_serve_wave: expert load");
      }
    }
    v.stamp[s] = now;
  }
  ++stats[ACCEPTMOE_POOL_WAVES];
  // routing of this wave's tokens rewritten to slots; other tokens route nowhere
  for (int t = 0; t < T; ++t) {
    const int32_t* row = topk_idx + static_cast<size_t>(t) * k;
    int32_t* out = slot_idx + static_cast<size_t>(t) * k;
    for (int j = 0; j < k; ++j) {
      const int e = row[j];
      bool first = e >= 0 && e < E;
      for (int q = 0; q < j && first; ++q) first = row[q] != e;
      out[j] = (wave_of[t] == wave && first) ? v.slot_of[e] : -1;
    }
  }
  return ACCEPTMOE_OK;
}

int32_t acceptmoe_copy_rows(const float* src, float* dst, const int32_t* row_tag, int32_t tag, int32_t T,
                            int32_t H, void* stream) {
  clear_err();
  if (T < 0 || H < 1) return fail(ACCEPTMOE_ERR_INVALID_ARG, "copy_rows: bad sizes (T=%d H=%d)", T, H);
  if (H % 4 != 0 || T > 65535)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "copy_rows: need H %% 4 == 0 and T <= 65535 (T=%d H=%d)", T, H);
  if (T == 0) return ACCEPTMOE_OK;
  if (!src || !dst || !row_tag) return fail(ACCEPTMOE_ERR_INVALID_ARG, "copy_rows: null pointer");
  if (!aligned(src, 16) || !aligned(dst, 16)) return fail(ACCEPTMOE_ERR_INVALID_ARG, "copy_rows: src and dst must be 16-byte aligned");
  hipError_t e = amoe::launch_copy_rows(src, dst, row_tag, tag, T, H, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ACCEPTMOE_OK : hip_fail(e, "copy_rows launch");
}

}  // extern "C"
