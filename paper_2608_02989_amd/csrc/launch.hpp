// Host-side launch functions of the kernels (internal to the library; the
// public boundary is include/acceptmoe.h).  Each returns the HIP status of
// its launches.  Arguments are already validated by the API layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace amoe {

constexpr int kMaxTrees = 256;
constexpr int kMaxTreeNodes = 1024;
constexpr int kMaxExperts = 512;
constexpr int kMaxTopK = 32;
constexpr int kNumStats = 10;

// ---- router (route.hip) ----
size_t packed_router_bytes(int E, int H);
hipError_t launch_pack_router(const float* src, int E, int H, void* dst, hipStream_t stream);
hipError_t launch_route(const void* hidden, int hidden_is_bf16, const void* router_packed, int T, int H,
                        int E, float* logits, hipStream_t stream);

// ---- selection (select.hip) ----
struct TreeOffsets {
  int32_t o[kMaxTrees + 1];
};

struct SelectParams {
  const float* logits;
  const int32_t* parent;
  const int32_t* depth;
  const float* prob;
  const uint8_t* resident;
  uint8_t* eligible;
  int32_t* topk_idx;
  float* topk_gate;
  int32_t* stats;
  int32_t* ws_kidx;    // [T, k] natural top-k experts (slot order)
  double* ws_r;        // [T, k] their router probabilities r_{t,e} (fp64)
  double* ws_rfull;    // [T, E] full softmax rows (MoE-Spec mass only)
  uint32_t* ws_routed; // [B, kMaxExperts / 32] experts that received a node of tree b
  double beta;
  int T, E, k, B, mode, budget, removal_cap;
};

size_t select_workspace_bytes(int T, int E, int k);
// host checks of acceptmoe_select and its allocation-free variant (api.cpp);
// returns an acceptmoe status, sets noop for an empty call
int32_t select_prepare(const char* who, const float* logits, const int32_t* parent, const int32_t* depth,
                       const float* commit_prob, const int32_t* tree_offsets, int32_t B, int32_t T, int32_t E,
                       int32_t k, double beta, int32_t mode, int32_t budget, int32_t removal_cap,
                       const uint8_t* resident_mask, uint8_t* eligible, int32_t* topk_idx, float* topk_gate,
                       int32_t* stats, SelectParams& p, TreeOffsets& offs, bool& noop);
void select_carve(void* ws, int T, int E, int k, SelectParams& p);
hipError_t launch_select(const SelectParams& p, const TreeOffsets& offs, hipStream_t stream);
hipError_t launch_commit_expand(const float* p_hat, int D, const int32_t* depth, int T, float* prob,
                                hipStream_t stream);

// ---- expert FFN (forward.hip) ----
hipError_t launch_pack(const void* src, int is_bf16, int E, int N, int K, void* dst, hipStream_t stream);
size_t packed_gate_up_bytes(int is_bf16, int E, int I, int H);
hipError_t launch_residual_add(const void* hidden, int is_bf16, const float* y, int T, int H, void* out,
                               hipStream_t stream);
hipError_t launch_copy_rows(const float* src, float* dst, const int32_t* row_tag, int tag, int T, int H,
                            hipStream_t stream);
hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t* sink, int grid, hipStream_t stream);
hipError_t launch_pack_gate_up(const void* gate, const void* up, int is_bf16, int E, int I, int H, void* dst,
                               hipStream_t stream);

struct ForwardParams {
  const void* hidden;
  const void* w_gate_up;  // packed gate/up tile pairs
  const void* w_down;
  const int32_t* topk_idx;
  const float* topk_gate;
  float* out;
  // workspace
  int32_t* cnt;       // [E]
  int32_t* off;       // [E + 1]
  int32_t* active;    // [E]
  int32_t* n_active;  // [1]
  int32_t* ent_slot;  // [T * k] slot ids grouped by expert, token order
  void* act;          // [T * k, I] bf16 or fp32
  float* ys;          // [T * k, H] gate-weighted expert outputs (per-slot down pass only)
  int4* items;        // down-pass work items (e, first CSR row, rows) (column-tile pass only)
  int32_t* n_items;   // [1]
  int T, H, I, E, k, is_bf16;
  int zero_out;       // gate/up pass clears out (the down pass then adds two halves into it)
  int item_rows;      // tokens per column-tile down item (16 per M-tile)
};

size_t forward_workspace_bytes(int T, int H, int I, int E, int k, int is_bf16);
void forward_carve(void* ws, ForwardParams& p);
hipError_t launch_forward(ForwardParams p, hipStream_t stream);

}  // namespace amoe
