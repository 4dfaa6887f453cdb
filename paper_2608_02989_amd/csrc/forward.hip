// Grouped SwiGLU expert FFN over the restricted routing (Sec. 3.1, Eq. 2):
// only experts that receive a token are streamed, each exactly once.
//
//   dispatch   one workgroup: per-expert token lists in node order (CSR) and
//              the list of active experts
//   gate_up    per (active expert, 16-row tile of I): X_e W_g^T and X_e W_u^T on
//              MFMA (tokens on the 16-wide M side), SwiGLU in registers, the
//              activation written once
//   down       blocks of up to kColMaxT tokens: per 16-column tile of H (and
//              half of I), act_e W_d^T for every dispatched (expert, 16-token
//              block), scaled by the gates and summed per token in LDS, then
//              written to out -- no per-slot buffer, no combine pass.
//              Larger blocks: per (active expert, 16-row tile of H), scaled
//              rows to the token's slot row, then
//   combine    out_t = sum over the k slots of token t, in slot order
//
// Weights are read in the packed fragment layout (see
// acceptmoe_pack_expert_weights): one wave load = one contiguous 1 KiB block.
#include <type_traits>

#include "common.hpp"
#include "launch.hpp"

namespace amoe {

namespace {

constexpr int kDispatchThreads = 1024;
constexpr int kDispatchChunk = kDispatchThreads;  // nodes per bitmask pass (one per thread)

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// ---------------------------------------------------------------------------
// weight packing: [E, N, K] row-major -> [E][N/16][K/KF][64 lanes][16 B]
// ---------------------------------------------------------------------------
__global__ void pack_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, int E, int N,
                            int rowbytes) {
  const int chunks_per_row = rowbytes / 64;  // 64-byte K chunks per row
  const size_t total = static_cast<size_t>(E) * N * chunks_per_row * 4;  // 16-B pieces
  for (size_t c = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; c < total;
       c += static_cast<size_t>(gridDim.x) * blockDim.x) {
    const int lane = static_cast<int>(c & 63);
    size_t f = c >> 6;  // fragment index = ((e * NT) + nt) * KC + kc
    const int kc = static_cast<int>(f % chunks_per_row);
    f /= chunks_per_row;
    const int nt = static_cast<int>(f % (N / 16));
    const int e = static_cast<int>(f / (N / 16));
    const int row = nt * 16 + (lane & 15);
    const size_t byte = (static_cast<size_t>(e) * N + row) * rowbytes + kc * 64 + (lane >> 4) * 16;
    dst[c] = src[byte / 16];
  }
}

// gate and up stacks [E, I, H] -> [E][I/32 tile pairs][K/KF][4][64 lanes][16 B]:
// fragments gate 2p, gate 2p+1, up 2p, up 2p+1 of each K chunk side by side;
// the second tile of the last pair is zero when I/16 is odd.
__global__ void pack_gate_up_kernel(const uint4* __restrict__ gate, const uint4* __restrict__ up,
                                    uint4* __restrict__ dst, int E, int I, int rowbytes) {
  const int chunks_per_row = rowbytes / 64;
  const int npairs = (I / 16 + 1) / 2;
  const size_t total = static_cast<size_t>(E) * npairs * chunks_per_row * 4 * 64;  // 16-B pieces
  for (size_t c = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; c < total;
       c += static_cast<size_t>(gridDim.x) * blockDim.x) {
    const int lane = static_cast<int>(c & 63);
    const int f = static_cast<int>((c >> 6) & 3);
    size_t q = c >> 8;
    const int kc = static_cast<int>(q % chunks_per_row);
    q /= chunks_per_row;
    const int pair = static_cast<int>(q % npairs);
    const int e = static_cast<int>(q / npairs);
    const int row = (2 * pair + (f & 1)) * 16 + (lane & 15);
    const uint4* src = (f >> 1) ? up : gate;
    dst[c] = row < I ? src[((static_cast<size_t>(e) * I + row) * rowbytes + kc * 64 + (lane >> 4) * 16) / 16]
                     : make_uint4(0u, 0u, 0u, 0u);
  }
}

// A node's routing row, loaded once: experts e[j] and a bit per slot that
// takes part in the dispatch.  A slot is skipped when its index lies outside
// [0, E) or repeats the expert of an earlier slot of the same node (a repeated
// expert is used once, at its first slot).
template <int KMAX>
__device__ __forceinline__ uint32_t load_route_row(const int32_t* __restrict__ row, int k, int E,
                                                   int (&e)[KMAX]) {
#pragma unroll
  for (int j = 0; j < KMAX; ++j) e[j] = j < k ? row[j] : -1;
  uint32_t valid = 0u;
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    bool ok = (e[j] >= 0) & (e[j] < E);
#pragma unroll
    for (int j2 = 0; j2 < j; ++j2) ok = ok & (e[j2] != e[j]);
    valid |= ok ? (1u << j) : 0u;
  }
  return valid;
}

// Exclusive scan of per-expert counts and compaction of the active experts,
// in index order (one wave, lane = tid < 64).  Returns the number of active
// experts; off[E] = total dispatched slots.
__device__ __forceinline__ int scan_experts(const int* cnt, int* off, int* active, int* active_g, int E, int tid) {
  int base = 0, abase = 0;
  for (int e0 = 0; e0 < E; e0 += kWave) {
    const int e = e0 + tid;
    const int c = e < E ? cnt[e] : 0;
    const int incl = wave_incl_scan_i32(c);
    if (e < E) off[e] = base + incl - c;
    const uint64_t am = __ballot(c > 0);
    if (c > 0) {
      const int pos = abase + popc64(am & lanes_below(tid));
      active[pos] = e;
      if (active_g != nullptr) active_g[pos] = e;
    }
    abase += popc64(am);
    base += lane_value(incl, kWave - 1);
  }
  if (tid == 0) off[E] = base;
  return abase;
}

// Down-pass items (expert, first CSR row, rows) per block of p.item_rows
// tokens of each active expert, in active-expert order, and their count (one
// wave).
__device__ __forceinline__ void write_down_items(const ForwardParams& p, const int* cnt, const int* off,
                                                 const int* active, int na, int tid) {
  const int ir = p.item_rows;
  int base = 0;
  for (int a0 = 0; a0 < na; a0 += kWave) {
    const int a = a0 + tid;
    const int e = a < na ? active[a] : 0;
    const int c = a < na ? cnt[e] : 0;
    const int nb = (c + ir - 1) / ir;
    const int incl = wave_incl_scan_i32(nb);
    for (int m = 0; m < nb; ++m)
      p.items[base + incl - nb + m] = make_int4(e, off[e] + ir * m, min(ir, c - ir * m), 0);
    base += lane_value(incl, kWave - 1);
  }
  if (tid == 0) *p.n_items = base;
}

// ---------------------------------------------------------------------------
// dispatch: CSR of (expert -> slot ids in node order), active expert list.
// One workgroup; each thread owns one node per pass and keeps its row in
// registers.  Positions inside an expert's list come from per-expert node
// bitmasks, so the order is deterministic (node order).
// ---------------------------------------------------------------------------
template <int KMAX>
__global__ __launch_bounds__(kDispatchThreads) void dispatch_kernel(ForwardParams p) {
  __shared__ int s_cnt[kMaxExperts];
  __shared__ int s_off[kMaxExperts + 1];
  __shared__ int s_run[kMaxExperts];
  __shared__ int s_active[kMaxExperts];
  __shared__ int s_nact;
  __shared__ uint32_t s_mask[kMaxExperts * (kDispatchChunk / 32)];
  __shared__ int s_pre[kMaxExperts * (kDispatchChunk / 32)];  // nodes of e in the chunk's earlier words
  const int tid = threadIdx.x;
  const int E = p.E, k = p.k, T = p.T;
  constexpr int words = kDispatchChunk / 32;
  for (int e = tid; e < E; e += kDispatchThreads) {
    s_cnt[e] = 0;
    s_run[e] = 0;
  }
  __syncthreads();
  int ev[KMAX];
  uint32_t valid = 0u;
  for (int t = tid; t < T; t += kDispatchThreads) {
    valid = load_route_row<KMAX>(p.topk_idx + static_cast<size_t>(t) * k, k, E, ev);
#pragma unroll
    for (int j = 0; j < KMAX; ++j)
      if (valid & (1u << j)) atomicAdd(&s_cnt[ev[j]], 1);
  }
  __syncthreads();
  if (tid < kWave) {
    const int na = scan_experts(s_cnt, s_off, s_active, p.active, E, tid);
    if (tid == 0) {
      s_nact = na;
      *p.n_active = na;
    }
  }
  __syncthreads();
  if (p.items != nullptr && tid < kWave) write_down_items(p, s_cnt, s_off, s_active, s_nact, tid);
  for (int e = tid; e < E; e += kDispatchThreads) {
    p.cnt[e] = s_cnt[e];
    p.off[e] = s_off[e];
  }
  if (tid == 0) p.off[E] = s_off[E];
  // position of each slot inside its expert list = earlier nodes of that expert
  for (int t0 = 0; t0 < T; t0 += kDispatchChunk) {
    const int t = t0 + tid;
    for (int i = tid; i < E * words; i += kDispatchThreads) s_mask[i] = 0u;
    if (t < T && T > kDispatchChunk)
      valid = load_route_row<KMAX>(p.topk_idx + static_cast<size_t>(t) * k, k, E, ev);
    __syncthreads();
    if (t < T) {
#pragma unroll
      for (int j = 0; j < KMAX; ++j)
        if (valid & (1u << j)) atomicOr(&s_mask[ev[j] * words + (tid >> 5)], 1u << (tid & 31));
    }
    __syncthreads();
    // per expert, exclusive prefix of the word popcounts
    for (int e = tid; e < E; e += kDispatchThreads) {
      int c = 0;
      for (int w = 0; w < words; ++w) {
        s_pre[e * words + w] = c;
        c += __popc(s_mask[e * words + w]);
      }
    }
    __syncthreads();
    if (t < T) {
#pragma unroll
      for (int j = 0; j < KMAX; ++j) {
        if (valid & (1u << j)) {
          const int i = ev[j] * words + (tid >> 5);
          const int before = s_pre[i] + __popc(s_mask[i] & ((1u << (tid & 31)) - 1u));
          p.ent_slot[s_off[ev[j]] + s_run[ev[j]] + before] = t * k + j;
        }
      }
    }
    __syncthreads();
    for (int e = tid; e < E; e += kDispatchThreads) {
      const int i = e * words + words - 1;
      s_run[e] += s_pre[i] + __popc(s_mask[i]);
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// In-workgroup dispatch for blocks of up to kSelfMaxT tokens: every gate/up
// workgroup builds the same CSR in LDS from the routing rows (one row per
// thread), so no separate dispatch launch is needed; workgroup 0 also
// publishes it (and the down items) for the down pass.
// ---------------------------------------------------------------------------
constexpr int kSelfMaxT = 256;
constexpr int kSelfMaxSlots = 2048;
constexpr int kSelfWords = kSelfMaxT / 32;

struct SelfDispatch {
  int cnt[kMaxExperts];
  int off[kMaxExperts + 1];
  int active[kMaxExperts];
  uint32_t mask[kMaxExperts * kSelfWords];  // per-expert token bitmasks
  int ent[kSelfMaxSlots];                   // CSR: slot ids grouped by expert, token order
  int nact;
};

// blockDim.x == 256 >= T
template <int KMAX>
__device__ __forceinline__ void self_dispatch(const ForwardParams& p, SelfDispatch& sd, int tid) {
  const int E = p.E, k = p.k, T = p.T;
  const int words = (T + 31) / 32;
  // the routing row first, so its latency overlaps the LDS clearing
  int ev[KMAX];
  uint32_t valid = 0u;
  if (tid < T) valid = load_route_row<KMAX>(p.topk_idx + static_cast<size_t>(tid) * k, k, E, ev);
  for (int i = tid; i < E; i += 256) sd.cnt[i] = 0;
  for (int i = tid; i < E * words; i += 256) sd.mask[i] = 0u;
  __syncthreads();
  if (tid < T) {
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      if (valid & (1u << j)) {
        atomicAdd(&sd.cnt[ev[j]], 1);
        atomicOr(&sd.mask[ev[j] * words + (tid >> 5)], 1u << (tid & 31));
      }
    }
  }
  __syncthreads();
  if (tid < kWave) {
    const int na = scan_experts(sd.cnt, sd.off, sd.active, nullptr, E, tid);
    if (tid == 0) sd.nact = na;
  }
  __syncthreads();
  if (tid < T) {
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      if (valid & (1u << j)) {
        const uint32_t* m = sd.mask + ev[j] * words;
        int before = __popc(m[tid >> 5] & ((1u << (tid & 31)) - 1u));
        for (int w = 0; w < (tid >> 5); ++w) before += __popc(m[w]);
        sd.ent[sd.off[ev[j]] + before] = tid * k + j;
      }
    }
  }
  __syncthreads();
}

// Per-item dispatch of the gate/up pass: a workgroup needs only the expert of
// its item (the a-th routed expert in index order, from the block's routed
// mask), that expert's slot ids in node order, its count n_e and its first
// CSR row o_e (the dispatched slots of lower experts) -- a few ballots over
// the routing rows, so the weight stream starts early.
template <int KMAX>
struct ItemDispatch {
  uint32_t emask[kMaxExperts / 32];  // routed experts of the block
  int wcnt[4], wless[4];             // per wave: its tokens of e, its slots below e
  int ent[kSelfMaxT];                // slot ids of e (one per token at most)
  int row[kSelfMaxT][KMAX];          // routing rows, kept here rather than in registers
  uint32_t valid[kSelfMaxT];         // their dispatched slots (load_route_row)
};

// the a-th set bit of mask[0 .. words) (a < number of set bits)
__device__ __forceinline__ int nth_set_bit(const uint32_t* mask, int words, int a) {
  int w = 0;
  for (; w + 1 < words; ++w) {
    const int c = __popc(mask[w]);
    if (a < c) break;
    a -= c;
  }
  uint32_t m = mask[w];
  for (int i = 0; i < a; ++i) m &= m - 1u;  // drop the a lowest set bits
  return 32 * w + __builtin_ctz(m);
}

// CSR, active list and down items to the workspace
__device__ __forceinline__ void publish_dispatch(const ForwardParams& p, const SelfDispatch& sd, int tid) {
  const int E = p.E;
  for (int e = tid; e <= E; e += 256) {
    p.off[e] = sd.off[e];
    if (e < E) p.cnt[e] = sd.cnt[e];
  }
  for (int i = tid; i < sd.nact; i += 256) p.active[i] = sd.active[i];
  for (int i = tid; i < sd.off[E]; i += 256) p.ent_slot[i] = sd.ent[i];
  if (tid == 0) *p.n_active = sd.nact;
  if (tid < kWave) write_down_items(p, sd.cnt, sd.off, sd.active, sd.nact, tid);
}

// ---------------------------------------------------------------------------
// element-type traits for the two MFMA paths
// ---------------------------------------------------------------------------
struct Bf16Path {
  static constexpr int kElemBytes = 2;
  static constexpr int kKF = 32;  // K elements per 64-byte fragment row chunk
  // one 16x16x32 MFMA per fragment
  static __device__ __forceinline__ floatx4 mma(const uint4& a, const uint4& b, floatx4 c) {
    return mfma_bf16_16x16x32(a, b, c);
  }
};

struct F32Path {
  static constexpr int kElemBytes = 4;
  static constexpr int kKF = 16;
  // four 16x16x4 MFMAs per fragment; component j of lane (r, g) is K index 4g + j
  static __device__ __forceinline__ floatx4 mma(const uint4& a, const uint4& b, floatx4 c) {
    c = mfma_f32_16x16x4(__uint_as_float(a.x), __uint_as_float(b.x), c);
    c = mfma_f32_16x16x4(__uint_as_float(a.y), __uint_as_float(b.y), c);
    c = mfma_f32_16x16x4(__uint_as_float(a.z), __uint_as_float(b.z), c);
    c = mfma_f32_16x16x4(__uint_as_float(a.w), __uint_as_float(b.w), c);
    return c;
  }
};

__device__ __forceinline__ float silu_mul(float g, float u) { return g / (1.0f + __expf(-g)) * u; }

// Tunables (compile-time): k-steps per pipeline stage for small / large
// M-tile counts; per projection, the output tiles each wave computes on shared
// A fragments (NTW) and the number of waves splitting a tile's K range (KS).
#ifndef AMOE_KU_SMALL
#define AMOE_KU_SMALL 1
#endif
#ifndef AMOE_KU_LARGE
#define AMOE_KU_LARGE 1
#endif
#ifndef AMOE_GU_NTW
#define AMOE_GU_NTW 2
#endif
#ifndef AMOE_GU_KS
#define AMOE_GU_KS 4
#endif
// per-slot down pass (blocks of more than 256 tokens): four H-tiles per wave
// share each activation fragment, two waves split I (against two tiles and
// four waves: 1036 vs 1103 us for the whole forward at T = 512, H = 4096,
// I = 1536, where the activation reads had outweighed the weight reads)
#ifndef AMOE_DN_NTW
#define AMOE_DN_NTW 4
#endif
#ifndef AMOE_DN_KS
#define AMOE_DN_KS 2
#endif

// Weight streams.  Every weight fragment is read once per step, through a
// buffer load whose cache policy is chosen per pass: the gate/up stream is
// non-temporal; the down stream uses the default policy where H >= 4096 (two
// column tiles per workgroup, or the per-slot pass) and is non-temporal
// otherwise.  (Measured on the wide layer, H = 4096, I = 1536: the column-tile
// down pass takes 68.6 us with default-policy loads against 75.6 us
// non-temporal, the per-slot down pass at 512 tokens 375 against 396 us; the
// gate/up pass is fastest non-temporal, 601 against 612 us for plain global
// non-temporal loads and 621 us with the default policy.  At H = 2048 the
// default policy saves 0.8 us of the down pass but lets its weights evict the
// next layer's router planes from the Infinity Cache: the 48-layer pass ran
// 5027 against 4941 us per block.)  A weight run is addressed by a
// wave-uniform base and its length in bytes: a load past the run returns
// zero instead of reading other memory.
constexpr int kPolicyStream = 2;  // "nt": non-temporal
constexpr int kPolicyPlain = 0;   // default cache policy
constexpr int kBufferWord3 = 0x00020000;  // raw (untyped) buffer resource, 32-bit data format

// a pointer the whole wave holds, moved to scalar registers
__device__ __forceinline__ const uint4* uniform_ptr(const uint4* p) {
  const uint64_t u = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(u >> 32));
  return reinterpret_cast<const uint4*>((static_cast<uint64_t>(hi) << 32) | lo);
}

// 16-byte piece `piece` (lane included) of the run [base, base + bytes)
template <int kPolicy>
__device__ __forceinline__ uint4 load_weight(const uint4* base, int bytes, int piece) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  __amdgpu_buffer_rsrc_t r =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint4*>(base), static_cast<short>(0), bytes, kBufferWord3);
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, piece * 16, 0, kPolicy);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// k-steps per pipeline stage; two stages are kept in flight
template <int MT>
struct Stage {
  static constexpr int kU = MT <= 2 ? AMOE_KU_SMALL : AMOE_KU_LARGE;
};

// 16-byte LDS pieces per lane for the shared A stages of any pass with up to
// MTMAX M-tiles (two stages of kU * MT fragments)
template <int MTMAX>
constexpr int shared_a_pieces() {
  int best = 0;
  for (int mt = 1; mt <= MTMAX; ++mt) {
    const int ku = mt <= 2 ? AMOE_KU_SMALL : AMOE_KU_LARGE;
    best = ku * mt > best ? ku * mt : best;
  }
  return 2 * best;
}

// acc[nb][mt] += sum over the K chunks c_i = c_first + i * c_step, 0 <= i < n,
// of x[mt] (A, tokens) times w[nb] (B, weight rows).  w[nb] is the wave-uniform
// start of a weight run of wbytes bytes, in which chunk c's fragment sits at
// piece c * wstride + lane; x[mt] points at this lane's 16-byte piece of chunk
// 0 and chunk c sits c * 4 pieces further.  Loads run two stages ahead of the
// MFMAs and carry no branches, so the only waits are the in-order vmcnt
// waits on the stage being consumed.
template <class P, int MT, int NB, int kPolicy>
__device__ __forceinline__ void stream_tiles(const uint4* const (&w)[NB], int wbytes, const uint4* const (&x)[MT],
                                             int c_first, int c_step, int n, int wstride, floatx4 (&acc)[NB][MT]) {
  constexpr int kU = Stage<MT>::kU;
  const int lane = lane_id();
  uint4 wb0[kU][NB], wb1[kU][NB], xb0[kU][MT], xb1[kU][MT];
  auto load0 = [&](int i) {
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int c = c_first + (i + u) * c_step;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) wb0[u][nb] = load_weight<kPolicy>(w[nb], wbytes, c * wstride + lane);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) xb0[u][mt] = x[mt][c * 4];
    }
  };
  auto load1 = [&](int i) {
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int c = c_first + (i + u) * c_step;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) wb1[u][nb] = load_weight<kPolicy>(w[nb], wbytes, c * wstride + lane);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) xb1[u][mt] = x[mt][c * 4];
    }
  };
  auto comp0 = [&]() {
#pragma unroll
    for (int u = 0; u < kU; ++u)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[nb][mt] = P::mma(xb0[u][mt], wb0[u][nb], acc[nb][mt]);
  };
  auto comp1 = [&]() {
#pragma unroll
    for (int u = 0; u < kU; ++u)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[nb][mt] = P::mma(xb1[u][mt], wb1[u][nb], acc[nb][mt]);
  };
  // Steady state without branches: the prefetch of the next stage is issued
  // unconditionally before the current stage is consumed, so the wait-count
  // pass sees straight-line code and only waits for the stage being used.
  // The scheduling barriers keep the compiler from sinking a prefetch below
  // the MFMAs of the stage before it (which would drain the pipeline: the
  // waits for the current stage would then come before the next loads).
  // The last one or two stages are peeled off after the loop.
  const int nst = n / kU;
  if (nst > 0) {
    load0(0);
    int st = 0;
    for (; st + 2 < nst; st += 2) {
      load1((st + 1) * kU);
      __builtin_amdgcn_sched_barrier(0);
      comp0();
      load0((st + 2) * kU);
      __builtin_amdgcn_sched_barrier(0);
      comp1();
    }
    if (st + 1 < nst) {
      load1((st + 1) * kU);
      __builtin_amdgcn_sched_barrier(0);
      comp0();
      comp1();
    } else {
      comp0();
    }
  }
  for (int i = nst * kU; i < n; ++i) {
    const int c = c_first + i * c_step;
    uint4 wt[NB], xt[MT];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) wt[nb] = load_weight<kPolicy>(w[nb], wbytes, c * wstride + lane);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) xt[mt] = x[mt][c * 4];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[nb][mt] = P::mma(xt[mt], wt[nb], acc[nb][mt]);
  }
}

// acc[nb][mt] as in stream_tiles, for a workgroup whose 4 waves all cover the
// same K range: each A fragment of a stage is loaded from global memory once,
// by one of the 4 waves, into a double-buffered LDS stage and read from there
// by all of them.  Weight fragments stay per wave, two stages in flight.  All
// 4 waves must call this with the same kc range (it contains barriers).
template <class P, int MT, int NB, int kPolicy>
__device__ __forceinline__ void stream_tiles_shared(const uint4* const (&w)[NB], int wbytes,
                                                    const uint4* const (&x)[MT], int KC, int wstride,
                                                    floatx4 (&acc)[NB][MT], uint4* xs) {
  constexpr int kU = Stage<MT>::kU;
  constexpr int kFr = kU * MT;                   // A fragments per stage
  constexpr int kMine = (kFr + 3) / 4;           // of which this wave loads
  const int wave = wave_id(), lane = lane_id();
  // xs layout: [2 stages][kU][MT][64 lanes] 16-byte pieces
  auto xs_at = [&](int buf, int u, int mt) { return xs + ((buf * kU + u) * MT + mt) * kWave + lane; };
  uint4 wb0[kU][NB], wb1[kU][NB], ta[kMine];
  auto loadw0 = [&](int c) {
#pragma unroll
    for (int u = 0; u < kU; ++u)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) wb0[u][nb] = load_weight<kPolicy>(w[nb], wbytes, (c + u) * wstride + lane);
  };
  auto loadw1 = [&](int c) {
#pragma unroll
    for (int u = 0; u < kU; ++u)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) wb1[u][nb] = load_weight<kPolicy>(w[nb], wbytes, (c + u) * wstride + lane);
  };
  // fragment f of a stage (step f / MT, M-tile f % MT) is loaded by wave f % 4;
  // every index below is a compile-time constant, the wave test is uniform
  auto loada = [&](int c) {
#pragma unroll
    for (int f = 0; f < kFr; ++f)
      if ((f & 3) == wave) ta[f >> 2] = x[f % MT][(c + f / MT) * 4];
  };
  auto storea = [&](int buf) {
#pragma unroll
    for (int f = 0; f < kFr; ++f)
      if ((f & 3) == wave) *xs_at(buf, f / MT, f % MT) = ta[f >> 2];
  };
  auto comp = [&](int buf, uint4 (&wb)[kU][NB]) {
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      uint4 xa[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) xa[mt] = *xs_at(buf, u, mt);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[nb][mt] = P::mma(xa[mt], wb[u][nb], acc[nb][mt]);
    }
  };
  const int nst = KC / kU;  // full stages; a ragged tail follows
  if (nst > 0) {
    // stage st lives in LDS buffer st & 1 and registers wb0 / wb1; the
    // steady state is branch-free, the last one or two stages are peeled
    loadw0(0);
    loada(0);
    storea(0);
    __syncthreads();
    int st = 0;
    for (; st + 2 < nst; st += 2) {
      loadw1((st + 1) * kU);
      loada((st + 1) * kU);
      comp(0, wb0);
      storea(1);
      __syncthreads();
      loadw0((st + 2) * kU);
      loada((st + 2) * kU);
      comp(1, wb1);
      storea(0);
      __syncthreads();
    }
    if (st + 1 < nst) {
      loadw1((st + 1) * kU);
      loada((st + 1) * kU);
      comp(0, wb0);
      storea(1);
      __syncthreads();
      comp(1, wb1);
    } else {
      comp(0, wb0);
    }
    __syncthreads();  // the LDS stages may be reused by the next pass
  }
  for (int c = nst * kU; c < KC; ++c) {
    uint4 wt[NB], xt[MT];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) wt[nb] = load_weight<kPolicy>(w[nb], wbytes, c * wstride + lane);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) xt[mt] = x[mt][c * 4];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[nb][mt] = P::mma(xt[mt], wt[nb], acc[nb][mt]);
  }
}

// ---------------------------------------------------------------------------
// The two grouped projections share one pass structure.  A workgroup (4
// waves) owns a run of 16-row output tiles of one active expert.  Each wave
// computes NTW tiles that share its A fragments; the KS waves of a tile group
// split the K chunks round-robin (wave s takes chunks s, s + KS, ...; the
// group reads its weight run front to back together, which keeps the DRAM
// accesses of the whole chip in far fewer open rows than per-wave K ranges)
// and add their partial tiles in LDS in a fixed order (deterministic), so one
// workgroup covers 4 * NTW / KS tiles.
//   GateUp: rows of I, K = H, A = gathered hidden rows; each tile has a gate
//           and an up fragment; SwiGLU -> act (bf16 for the bf16 path, fp32
//           otherwise), written once per token row.  NTW = 2: the gate and up
//           fragments of a tile pair are adjacent in the packed layout
//           ([E][I/32][K chunk][gate 2p, gate 2p+1, up 2p, up 2p+1]), so a
//           K chunk of the pair is one 4 KiB run.
//   Down:   rows of H, K = I, A = act rows of the expert; gate-scaled rows go
//           to the token's slot row of ys.
// ---------------------------------------------------------------------------
enum class Proj { GateUp, Down };

template <Proj F, int NTW, int KS>
struct ProjShape {
  static constexpr int kNB = NTW * (F == Proj::GateUp ? 2 : 1);  // weight fragments per k-step
  static constexpr int kTilesPerWG = 4 * NTW / KS;
};

// ent_e: the n_e slot ids of expert e in node order; o_e: its first row in act
template <class P, Proj F, int MT, int NTW, int KS, int MG>
__device__ __forceinline__ void ffn_pass(const ForwardParams& p, const int32_t* ent_e, int e, int tile_base, int n_e,
                                         int o_e, int m0, floatx4 (*red)[kWave][4], uint4* xs) {
  static_assert(F != Proj::GateUp || NTW == 2, "the packed gate/up layout holds tile pairs");
  static_assert(KS % MG == 0, "M groups take waves from the K split");
  constexpr int NB = ProjShape<F, NTW, KS>::kNB;
  constexpr int KSe = KS / MG;  // waves per K split of one (tile group, M group)
  constexpr int TG = 4 / KS;    // tile groups per workgroup
  const int wave = wave_id(), lane = lane_id();
  const int r = lane & 15, g = lane >> 4;
  const int sub = wave % KSe;
  const int tile0 = tile_base + ((wave / KSe) % TG) * NTW;  // first of this wave's NTW tiles
  m0 += (wave / (KSe * TG)) * MT * 16;                      // this wave's M group
  const int ntiles = (F == Proj::GateUp ? p.I : p.H) / 16;
  const int K = F == Proj::GateUp ? p.H : p.I;
  const int KC = K / P::kKF;
  const int rowq = K * P::kElemBytes / 16;

  const uint4* x[MT];
  if (F == Proj::GateUp) {
    const uint4* hid = static_cast<const uint4*>(p.hidden);
    const int tok0 = ent_e[0] / p.k;  // rows past n_e read a valid row; their outputs are dropped
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = m0 + mt * 16 + r;
      const int tok = m < n_e ? ent_e[m] / p.k : tok0;
      x[mt] = hid + static_cast<size_t>(tok) * rowq + g;
    }
  } else {
    const uint4* act = static_cast<const uint4*>(p.act);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = m0 + mt * 16 + r;
      x[mt] = act + static_cast<size_t>(o_e + (m < n_e ? m : 0)) * rowq + g;
    }
  }
  // tiles past the end are clamped to a valid tile (pair): computed, never written
  const uint4* w[NB];  // wave-uniform starts of the weight runs
  int wstride;         // 16-byte pieces from one K chunk to the next
  int wbytes;          // bytes of each run from its start
  if (F == Proj::GateUp) {
    const int npairs = (ntiles + 1) / 2;
    const int pair = min(tile0 / 2, npairs - 1);
    const uint4* base = uniform_ptr(static_cast<const uint4*>(p.w_gate_up) +
                                    (static_cast<size_t>(e) * npairs + pair) * KC * 4 * kWave);
    w[0] = base;              // gate, tile 2 pair
    w[1] = base + 2 * kWave;  // up, tile 2 pair
    w[2] = base + kWave;      // gate, tile 2 pair + 1
    w[3] = base + 3 * kWave;  // up, tile 2 pair + 1
    wstride = 4 * kWave;
    wbytes = KC * 4 * kWave * 16 - 3 * kWave * 16;  // the last fragment of w[3] ends the pair's run
  } else {
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
      const int tile = min(tile0 + j, ntiles - 1);
      w[j] = uniform_ptr(static_cast<const uint4*>(p.w_down) + (static_cast<size_t>(e) * ntiles + tile) * KC * kWave);
    }
    wstride = kWave;
    wbytes = KC * kWave * 16;
  }
  constexpr int kPolicy = F == Proj::GateUp ? kPolicyStream : kPolicyPlain;
  floatx4 acc[NB][MT];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[nb][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
  if constexpr (KS == 1 && MG == 1)
    stream_tiles_shared<P, MT, NB, kPolicy>(w, wbytes, x, KC, wstride, acc, xs);
  else
    stream_tiles<P, MT, NB, kPolicy>(w, wbytes, x, sub, KSe, (KC - sub + KSe - 1) / KSe, wstride, acc);

  if constexpr (KSe > 1) {
    // fixed-order sum of the KS partial tiles, four fragments per LDS round
#pragma unroll
    for (int q0 = 0; q0 < NB * MT; q0 += 4) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (q0 + q < NB * MT) red[wave][lane][q] = acc[(q0 + q) / MT][(q0 + q) % MT];
      __syncthreads();
      if (sub == 0) {
#pragma unroll
        for (int s2 = 1; s2 < KSe; ++s2)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (q0 + q < NB * MT) {
              const floatx4 v = red[wave + s2][lane][q];
#pragma unroll
              for (int i = 0; i < 4; ++i) acc[(q0 + q) / MT][(q0 + q) % MT][i] += v[i];
            }
      }
      __syncthreads();
    }
  }
  if (sub == 0) {
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
      const int tile = tile0 + j;
      if (tile >= ntiles) continue;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + mt * 16 + 4 * g + i;
          if (m < n_e) {
            if (F == Proj::GateUp) {
              const float v = silu_mul(acc[2 * j][mt][i], acc[2 * j + 1][mt][i]);
              const size_t idx = static_cast<size_t>(o_e + m) * p.I + tile * 16 + r;
              if (P::kElemBytes == 2)
                static_cast<uint16_t*>(p.act)[idx] = float_to_bf16_bits(v);
              else
                static_cast<float*>(p.act)[idx] = v;
            } else {
              const int s = ent_e[m];
              p.ys[static_cast<size_t>(s) * p.H + tile * 16 + r] = p.topk_gate[s] * acc[j][mt][i];
            }
          }
        }
      }
    }
  }
}

// the full CSR is built only by the publishing workgroup, after its items
template <bool kSelf, int KMAX>
union SelfDispatchSlot {
  SelfDispatch sd;
  ItemDispatch<KMAX> id;
};
template <int KMAX>
union SelfDispatchSlot<false, KMAX> {
  int unused;
};

// Work item i = (active expert i / wg_per_expert, tile run i % wg_per_expert).
// Without kSelf: grid.x = cap_experts * wg_per_expert, one item per
// workgroup, reading dispatch_kernel's CSR.  kSelf (gate/up pass, blocks of up
// to kSelfMaxT tokens): a grid of up to kSelfGridMult times the workgroups
// resident at once (H >= 4096; once otherwise) takes items blockIdx.x,
// blockIdx.x + gridDim.x, ..., each with its own per-item dispatch.  The
// workgroups beyond the resident ones start on whichever CU frees a slot
// first, which evens out the CUs' finish times (CUs stream at up to 20 %
// different rates): at H = 4096, T = 64 the pass took 121.1 us with a
// resident-sized grid and 117.8 us with three times that.  The shorter items
// of H = 2048 (256 KiB) do not repay the prologue each extra workgroup
// repeats: the 48-layer pass at T = 60 ran 4951, 4990 and 5054 us per block
// with one, two and three times the resident grid.  Workgroups left without
// an item exit after the prologue.  Workgroup 0, which is dispatched first
// and has the most items, builds the full CSR afterwards and publishes it for
// the down pass.  (Claiming items from a device-wide counter was measured no
// better.)
constexpr int kSelfGridMult = 3;

// Occupancy floor: three workgroups per CU for up to two M-tiles, two for
// more (the register budget the streaming loop is tuned to).
template <class P, Proj F, int MTMAX, int NTW, int KS, bool kSelf, int KMAX>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(MTMAX <= 2 ? 3 : 2))) void ffn_kernel(
    ForwardParams p) {
  __shared__ floatx4 red[KS > 1 ? 4 : 1][kWave][4];
  __shared__ uint4 xs[KS == 1 ? shared_a_pieces<MTMAX>() * kWave : 1];
  __shared__ SelfDispatchSlot<kSelf, KMAX> sds;
  constexpr int tpw = ProjShape<F, NTW, KS>::kTilesPerWG;
  const int ntiles = (F == Proj::GateUp ? p.I : p.H) / 16;
  const int wg_per_expert = (ntiles + tpw - 1) / tpw;
  if (F == Proj::GateUp && p.zero_out) {
    // the column-tile down pass adds its two halves of I into out
    float4* o4 = reinterpret_cast<float4*>(p.out);
    const size_t n4 = static_cast<size_t>(p.T) * p.H / 4;
    for (size_t i = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n4;
         i += static_cast<size_t>(gridDim.x) * blockDim.x)
      o4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  // An expert with more than MTMAX M-tiles of tokens would stream its weights
  // once per MTMAX M-tiles.  Without the in-workgroup dispatch (blocks of more
  // than kSelfMaxT tokens) such an expert instead takes the waves of the K
  // split as M groups: MG = 2 or 4 groups of MT M-tiles each read the same
  // weight fragments (from L1 or L2 after the first), so the weights come
  // from HBM once per up to 4 MTMAX M-tiles.  At 512 tokens (8 trees of 64,
  // H = 4096) experts receive up to ~160 tokens and the forward took 1014.5
  // us with one pass per MTMAX M-tiles, 972.3 us with M groups.  Every wave
  // of the workgroup runs the same instantiation (the passes hold barriers).
  auto pass_mt = [&](auto mg_tag, int mt, int tile_base, int e, int n_e, int o_e, int m0, const int32_t* ent_e) {
    constexpr int G = decltype(mg_tag)::value;
    if (mt == 1) ffn_pass<P, F, 1, NTW, KS, G>(p, ent_e, e, tile_base, n_e, o_e, m0, red, xs);
    else if (MTMAX >= 2 && mt == 2) ffn_pass<P, F, (MTMAX >= 2 ? 2 : 1), NTW, KS, G>(p, ent_e, e, tile_base, n_e, o_e, m0, red, xs);
    else if (MTMAX >= 3 && mt == 3) ffn_pass<P, F, (MTMAX >= 3 ? 3 : 1), NTW, KS, G>(p, ent_e, e, tile_base, n_e, o_e, m0, red, xs);
    else ffn_pass<P, F, MTMAX, NTW, KS, G>(p, ent_e, e, tile_base, n_e, o_e, m0, red, xs);
  };
  auto run_expert = [&](int tile_base, int e, int n_e, int o_e, const int32_t* ent_e) {
    for (int m0 = 0; m0 < n_e;) {
      const int left = (n_e - m0 + 15) / 16;  // M-tiles still to cover
      if (kSelf || left <= MTMAX || KS % 2 != 0) {
        const int mt = min(MTMAX, left);
        pass_mt(std::integral_constant<int, 1>{}, mt, tile_base, e, n_e, o_e, m0, ent_e);
        m0 += 16 * mt;
      } else if (KS % 4 == 0 && left > 2 * MTMAX) {
        const int mt = (min(left, 4 * MTMAX) + 3) / 4;
        pass_mt(std::integral_constant<int, (KS % 4 == 0 ? 4 : 1)>{}, mt, tile_base, e, n_e, o_e, m0, ent_e);
        m0 += 64 * mt;
      } else {
        const int mt = (min(left, 2 * MTMAX) + 1) / 2;
        pass_mt(std::integral_constant<int, (KS % 2 == 0 ? 2 : 1)>{}, mt, tile_base, e, n_e, o_e, m0, ent_e);
        m0 += 32 * mt;
      }
    }
  };
  if constexpr (kSelf) {
    ItemDispatch<KMAX>& id = sds.id;
    const int tid = threadIdx.x, wave = wave_id(), lane = lane_id();
    const int T = p.T, k = p.k, E = p.E, words = (E + 31) / 32;
    if (tid < kMaxExperts / 32) id.emask[tid] = 0u;
    {
      int ev[KMAX];
#pragma unroll
      for (int j = 0; j < KMAX; ++j) ev[j] = -1;
      uint32_t valid = 0u;
      if (tid < T) {
        valid = load_route_row<KMAX>(p.topk_idx + static_cast<size_t>(tid) * k, k, E, ev);
#pragma unroll
        for (int j = 0; j < KMAX; ++j) id.row[tid][j] = ev[j];
        id.valid[tid] = valid;
      }
      __syncthreads();
#pragma unroll
      for (int j = 0; j < KMAX; ++j)
        if (valid & (1u << j)) atomicOr(&id.emask[ev[j] >> 5], 1u << (ev[j] & 31));
    }
    __syncthreads();
    // workgroup-uniform values go to scalar registers (the streaming loop
    // needs every vector register it can get)
    int nact = 0;
    for (int w = 0; w < words; ++w) nact += __popc(id.emask[w]);
    nact = __builtin_amdgcn_readfirstlane(nact);
    const int n_items = nact * wg_per_expert;
    for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
      const int e = __builtin_amdgcn_readfirstlane(nth_set_bit(id.emask, words, item / wg_per_expert));
      // this thread's token: its slot of e, and its slots of lower experts
      int slot = -1, less = 0;
      if (tid < T) {
        const uint32_t valid = id.valid[tid];
#pragma unroll
        for (int j = 0; j < KMAX; ++j) {
          const int ej = id.row[tid][j];
          if (valid & (1u << j)) {
            slot = ej == e ? static_cast<int>(tid) * k + j : slot;
            less += ej < e ? 1 : 0;
          }
        }
      }
      const uint64_t hm = __ballot(slot >= 0);
      const int wless = wave_sum_i32(less);
      __syncthreads();  // the previous item's list is no longer read
      if (lane == 0) {
        id.wcnt[wave] = popc64(hm);
        id.wless[wave] = wless;
      }
      __syncthreads();
      int before = 0, n_e = 0, o_e = 0;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        before += w < wave ? id.wcnt[w] : 0;
        n_e += id.wcnt[w];
        o_e += id.wless[w];
      }
      if (slot >= 0) id.ent[before + popc64(hm & lanes_below(lane))] = slot;
      __syncthreads();
      run_expert((item % wg_per_expert) * tpw, e, __builtin_amdgcn_readfirstlane(n_e),
                 __builtin_amdgcn_readfirstlane(o_e), id.ent);
    }
    if (blockIdx.x == 0) {
      __syncthreads();  // the per-item state shares this LDS
      SelfDispatch& sd = sds.sd;
      self_dispatch<KMAX>(p, sd, tid);
      publish_dispatch(p, sd, tid);
    }
  } else {
    if (static_cast<int>(blockIdx.x) >= *p.n_active * wg_per_expert) return;
    const int a = blockIdx.x / wg_per_expert;
    const int e = p.active[a];
    run_expert((blockIdx.x % wg_per_expert) * tpw, e, p.cnt[e], p.off[e], p.ent_slot + p.off[e]);
  }
}

// ---------------------------------------------------------------------------
// Column-tile down pass (blocks of up to kColMaxT tokens).  A workgroup owns
// NB adjacent 16-column tiles of H and one of `ksplit` (1 or 2) parts of I.
// It streams those tiles' rows of W_d for every down item (expert e, block of
// up to 16 MTI tokens of e's list): the items are dealt round-robin to the
// waves, and each wave runs one continuous two-stage load pipeline across its
// items.  The MTI M-tiles of an item share every weight fragment, so an
// expert's slice of W_d is streamed once per 16 MTI tokens (an expert with 17
// to 32 tokens took two passes over it with 16-token items; the second mostly
// from L2, yet the pass ran at 4.6 instead of 5.9 TB/s).  A second M-tile with
// no token reads a valid row again (a cache hit); its products are dropped.
// After an item's last stage the wave adds gate * (act_e W_d^T) into its own
// LDS accumulator out_w[t, 16 NB columns] (a token appears once per expert, so
// the lanes of one item never collide).  At the end the waves' accumulators are
// summed in wave order and written to out, or added into the zeroed out when
// I is split in two (two fp32 additions onto zero commute, so the result
// does not depend on which half lands first).  Every workgroup does the same
// work; its LDS footprint keeps it alone on its CU.  Each workgroup reads
// every dispatched activation row once, so NB = 2 halves that traffic per
// column for wide H.
// ---------------------------------------------------------------------------
constexpr int kColLanes = 8;  // waves x NB: the accumulators take kColLanes x kColMaxT x 16 floats
constexpr int kColMaxT = 256;
constexpr int kColMaxSlots = 2048;
constexpr int kColMaxItems = kMaxExperts + kColMaxSlots / 16;

struct ColShared {
  float acc[kColLanes * kColMaxT * 16];  // per-wave token accumulators [wave][t][16 NB]
  int tok[kColMaxSlots];                 // CSR row -> token
  float gw[kColMaxSlots];                // CSR row -> gate of that slot
  int4 items[kColMaxItems];
};

template <class P, int kU, int NB, int MTI>
__global__ __launch_bounds__(kColLanes / NB * kWave) void down_col_kernel(ForwardParams p, int ksplit) {
  constexpr int kWaves = kColLanes / NB;
  constexpr int kThreads = kWaves * kWave;
  constexpr int kCols = 16 * NB;
  __shared__ ColShared sh;
  const int tid = threadIdx.x;
  const int wave = wave_id(), lane = lane_id();
  const int r = lane & 15, g = lane >> 4;
  const int T = p.T, H = p.H, k = p.k;
  const int ntiles = H / 16;
  const int ngroups = ntiles / NB;
  const int ht0 = (blockIdx.x % ngroups) * NB, part = blockIdx.x / ngroups;
  const int KC = p.I / P::kKF;
  const int kc0 = part * KC / ksplit;
  const int L = (KC / ksplit) / kU;  // pipeline stages per item
  const int rowq = p.I * P::kElemBytes / 16;
  const int n_items = *p.n_items;
  const int n_rows = p.off[p.E];
  // this wave's first item straight from the workspace, so the first stage's
  // loads are in flight while the lists are staged in LDS
  int4 first = make_int4(0, 0, 1, 0);
  if (wave < n_items) first = p.items[wave];
  for (int i = tid; i < kWaves * T * kCols; i += kThreads) sh.acc[i] = 0.f;
  for (int i = tid; i < n_rows; i += kThreads) {
    const int slot = p.ent_slot[i];
    sh.tok[i] = slot / k;
    sh.gw[i] = p.topk_gate[slot];
  }
  for (int i = tid; i < n_items; i += kThreads) sh.items[i] = p.items[i];

  const uint4* wd = static_cast<const uint4*>(p.w_down);
  const uint4* act = static_cast<const uint4*>(p.act);
  float* accw = sh.acc + wave * T * kCols;
  // items wave, wave + kWaves, ...; stage = (item, q), q in [0, L)
  const int my_items = n_items > wave ? (n_items - wave + kWaves - 1) / kWaves : 0;
  const int nst = my_items * L;
  struct Cursor {
    int it, q, e, row0, nrows;
  };
  auto fetch = [&](Cursor& c) {
    if (c.it < n_items) {
      const int4 d = sh.items[c.it];
      c.e = d.x;
      c.row0 = d.y;
      c.nrows = d.z;
    }
  };
  auto advance = [&](Cursor& c) {
    if (++c.q == L) {
      c.q = 0;
      c.it += kWaves;
      fetch(c);
    }
  };
  uint4 w0[kU][NB], x0[kU][MTI], w1[kU][NB], x1[kU][MTI];
  auto load = [&](uint4 (&wv)[kU][NB], uint4 (&xv)[kU][MTI], const Cursor& c) {
    const int kc = kc0 + c.q * kU;
    const uint4* xp[MTI];
#pragma unroll
    for (int mt = 0; mt < MTI; ++mt)
      xp[mt] = act + static_cast<size_t>(c.row0 + min(16 * mt + r, c.nrows - 1)) * rowq + g + kc * 4;
    const uint4* wrun = uniform_ptr(wd + (static_cast<size_t>(c.e) * ntiles + ht0) * KC * kWave);
#pragma unroll
    for (int u = 0; u < kU; ++u) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        wv[u][nb] = load_weight<NB == 2 ? kPolicyPlain : kPolicyStream>(wrun, NB * KC * kWave * 16,
                                                                        (nb * KC + kc + u) * kWave + lane);
#pragma unroll
      for (int mt = 0; mt < MTI; ++mt) xv[u][mt] = xp[mt][u * 4];
    }
  };
  floatx4 acc[NB][MTI];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int mt = 0; mt < MTI; ++mt) acc[nb][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](uint4 (&wv)[kU][NB], uint4 (&xv)[kU][MTI], Cursor& c) {
#pragma unroll
    for (int u = 0; u < kU; ++u)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int mt = 0; mt < MTI; ++mt) acc[nb][mt] = P::mma(xv[u][mt], wv[u][nb], acc[nb][mt]);
    if (c.q == L - 1) {
      // item done: out_w[t] += gate * row, rows 16 mt + 4g .. +3 of the item, column r of each tile
#pragma unroll
      for (int mt = 0; mt < MTI; ++mt) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = 16 * mt + 4 * g + i;
          if (m < c.nrows) {
            const int row = c.row0 + m;
            float* dst = accw + sh.tok[row] * kCols + r;
            const float gt = sh.gw[row];
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) dst[16 * nb] += gt * acc[nb][mt][i];
          }
        }
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int mt = 0; mt < MTI; ++mt) acc[nb][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
    advance(c);
  };
  Cursor lc{wave, 0, first.x, first.y, first.z}, cc{wave, 0, first.x, first.y, first.z};
  if (nst > 0) load(w0, x0, lc);
  __syncthreads();  // lists staged, accumulators cleared (advance reads the staged items)
  if (nst > 0) {
    advance(lc);
    int st = 0;
    for (; st + 2 < nst; st += 2) {
      load(w1, x1, lc);
      advance(lc);
      compute(w0, x0, cc);
      load(w0, x0, lc);
      advance(lc);
      compute(w1, x1, cc);
    }
    if (st + 1 < nst) {
      load(w1, x1, lc);
      compute(w0, x0, cc);
      compute(w1, x1, cc);
    } else {
      compute(w0, x0, cc);
    }
  }
  __syncthreads();
  // fixed-order sum over the waves, then out (or out += for a half of I)
  for (int i = tid; i < T * kCols; i += kThreads) {
    float v = sh.acc[i];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) v += sh.acc[w * T * kCols + i];
    float* o = p.out + static_cast<size_t>(i / kCols) * H + ht0 * 16 + (i % kCols);
    if (ksplit == 2) atomicAdd(o, v);
    else *o = v;
  }
}

// ---------------------------------------------------------------------------
// combine: out[t, h] = sum over the dispatched slots of token t, in slot order.
// The routing row and all k expert rows are loaded before any is used (rows
// of skipped slots are read but discarded).  Workgroup b covers token
// b / hblocks, float4 columns 256 (b % hblocks) ..; a one-dimensional grid, so
// any T fits.
// ---------------------------------------------------------------------------
template <int KMAX>
__global__ __launch_bounds__(256) void combine_kernel(ForwardParams p, int hblocks) {
  const int t = blockIdx.x / hblocks;
  const int h4 = (blockIdx.x % hblocks) * blockDim.x + threadIdx.x;  // float4 column
  const int H = p.H, k = p.k;
  if (h4 * 4 >= H) return;
  int ev[KMAX];
  const uint32_t valid = load_route_row<KMAX>(p.topk_idx + static_cast<size_t>(t) * k, k, p.E, ev);
  float4 v[KMAX];
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    const int jj = j < k ? j : k - 1;
    v[j] = reinterpret_cast<const float4*>(p.ys + (static_cast<size_t>(t) * k + jj) * H)[h4];
  }
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    if (valid & (1u << j)) {
      s.x += v[j].x;
      s.y += v[j].y;
      s.z += v[j].z;
      s.w += v[j].w;
    }
  }
  reinterpret_cast<float4*>(p.out + static_cast<size_t>(t) * H)[h4] = s;
}

// Workgroups of kernel `Kern` (256 threads) resident on the current device at
// once, computed on first use per kernel and device (a template per kernel, so
// kernels of different register or LDS needs keep separate counts).
template <auto Kern>
int resident_workgroups() {
  constexpr int kMaxDevices = 64;
  static int cached[kMaxDevices] = {};
  const auto kernel = Kern;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) dev = 0;
  if (cached[dev] == 0) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, 256, 0) != hipSuccess || per_cu < 1) per_cu = 1;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) cus = 1;
    cached[dev] = per_cu * cus;
  }
  return cached[dev];
}

template <class P, int MTMAX>
hipError_t launch_gate_up(const ForwardParams& p, int cap, bool self, hipStream_t stream) {
  constexpr int gt = ProjShape<Proj::GateUp, AMOE_GU_NTW, AMOE_GU_KS>::kTilesPerWG;
  const int items = cap * ((p.I / 16 + gt - 1) / gt);
  if (!self) {
    ffn_kernel<P, Proj::GateUp, MTMAX, AMOE_GU_NTW, AMOE_GU_KS, false, 8><<<dim3(items), 256, 0, stream>>>(p);
  } else if (p.k <= 8) {
    constexpr auto kern = &ffn_kernel<P, Proj::GateUp, MTMAX, AMOE_GU_NTW, AMOE_GU_KS, true, 8>;
    const int res = (p.H >= 4096 ? kSelfGridMult : 1) * resident_workgroups<kern>();
    kern<<<dim3(items < res ? items : res), 256, 0, stream>>>(p);
  } else {
    constexpr auto kern = &ffn_kernel<P, Proj::GateUp, MTMAX, AMOE_GU_NTW, AMOE_GU_KS, true, kMaxTopK>;
    const int res = (p.H >= 4096 ? kSelfGridMult : 1) * resident_workgroups<kern>();
    kern<<<dim3(items < res ? items : res), 256, 0, stream>>>(p);
  }
  return hipGetLastError();
}

template <class P, int MTMAX>
hipError_t launch_down_rows(const ForwardParams& p, int cap, hipStream_t stream) {
  constexpr int dt = ProjShape<Proj::Down, AMOE_DN_NTW, AMOE_DN_KS>::kTilesPerWG;
  const int dn_wg = (p.H / 16 + dt - 1) / dt;
  ffn_kernel<P, Proj::Down, MTMAX, AMOE_DN_NTW, AMOE_DN_KS, false, 8><<<dim3(cap * dn_wg), 256, 0, stream>>>(p);
  return hipGetLastError();
}

// Column-tile down pass shape: I split in two when that keeps the grid near
// 256 workgroups, two column tiles per workgroup for wide H, k-steps per
// pipeline stage: the largest of 12, 8, 6, 4, 3, 2, 1 dividing the part of I,
// at most 12 with one column tile (two stages in flight then fit the
// registers of one 8-wave workgroup per CU, and the deeper stages keep more
// bytes in flight: 12 vs 4 k-steps measured 0.6 us faster at H = 2048,
// I = 768) and at most 4 with two (whose stages already carry twice the
// weight bytes; 8 measured slower at H = 4096, I = 1536).  Thin parts of I
// (one GPU's share of a tensor-parallel split) give lengths like 3, where
// 3-step stages ran 11 % faster than single steps.
struct ColShape {
  int ksplit, ku, nb, mti;
};

#ifndef AMOE_COL_MTI
#define AMOE_COL_MTI 0
#endif

// M-tiles per down item: two (items of up to 32 tokens) for blocks of more
// than 32 tokens when the workgroup owns two column tiles, whose stages are
// capped at 4 k-steps either way (H = 4096, T = 64: forward 188.7 -> 182.9 us);
// with one column tile a second M-tile would halve the 12-k-step stages, which
// cost more than it saves where experts receive ~10 tokens (H = 2048, T = 60:
// 48-layer pass 4926 -> 5063 us per block).
ColShape col_shape(int T, int H, int I, int is_bf16) {
  const int KC = I / (is_bf16 ? Bf16Path::kKF : F32Path::kKF);
  const int ntiles = H / 16;
  ColShape c;
  c.nb = (ntiles >= 256 && ntiles % 2 == 0) ? 2 : 1;
  c.mti = AMOE_COL_MTI ? AMOE_COL_MTI : (T > 32 && c.nb == 2 ? 2 : 1);
  c.ksplit = (ntiles / c.nb <= 128 && KC % 2 == 0) ? 2 : 1;
  const int len = KC / c.ksplit;
  const int ku_max = c.nb == 1 ? (c.mti == 1 ? 12 : 6) : 4;
  c.ku = 1;
  for (const int u : {12, 8, 6, 4, 3, 2}) {
    if (len % u == 0 && u <= ku_max) {
      c.ku = u;
      break;
    }
  }
  return c;
}

// blocks of up to 256 tokens and 2048 slots: gate/up builds its own dispatch,
// the column-tile down pass replaces the per-slot pass and combine
bool use_col_path(int T, int k) {
  return T <= kColMaxT && T <= kSelfMaxT && static_cast<long long>(T) * k <= kColMaxSlots &&
         static_cast<long long>(T) * k <= kSelfMaxSlots;
}

template <class P, int NB, int MTI>
hipError_t launch_down_col_nb(const ForwardParams& p, const ColShape& c, hipStream_t stream) {
  const dim3 grid((p.H / 16 / NB) * c.ksplit);
  constexpr int threads = kColLanes / NB * kWave;
  if constexpr (NB == 1) {  // deeper stages only with one column tile (col_shape)
    if constexpr (MTI == 1) {
      if (c.ku == 12 || c.ku == 8) {
        if (c.ku == 12) down_col_kernel<P, 12, NB, MTI><<<grid, threads, 0, stream>>>(p, c.ksplit);
        else down_col_kernel<P, 8, NB, MTI><<<grid, threads, 0, stream>>>(p, c.ksplit);
        return hipGetLastError();
      }
    }
    if (c.ku == 6) {
      down_col_kernel<P, 6, NB, MTI><<<grid, threads, 0, stream>>>(p, c.ksplit);
      return hipGetLastError();
    }
  }
  if (c.ku == 4) down_col_kernel<P, 4, NB, MTI><<<grid, threads, 0, stream>>>(p, c.ksplit);
  else if (c.ku == 3) down_col_kernel<P, 3, NB, MTI><<<grid, threads, 0, stream>>>(p, c.ksplit);
  else if (c.ku == 2) down_col_kernel<P, 2, NB, MTI><<<grid, threads, 0, stream>>>(p, c.ksplit);
  else down_col_kernel<P, 1, NB, MTI><<<grid, threads, 0, stream>>>(p, c.ksplit);
  return hipGetLastError();
}

template <class P>
hipError_t launch_down_col(const ForwardParams& p, const ColShape& c, hipStream_t stream) {
  if (c.mti == 2)
    return c.nb == 2 ? launch_down_col_nb<P, 2, 2>(p, c, stream) : launch_down_col_nb<P, 1, 2>(p, c, stream);
  return c.nb == 2 ? launch_down_col_nb<P, 2, 1>(p, c, stream) : launch_down_col_nb<P, 1, 1>(p, c, stream);
}

}  // namespace

size_t packed_gate_up_bytes(int is_bf16, int E, int I, int H) {
  return static_cast<size_t>(E) * ((I / 16 + 1) / 2) * 32 * H * (is_bf16 ? 2 : 4) * 2;
}

hipError_t launch_pack_gate_up(const void* gate, const void* up, int is_bf16, int E, int I, int H, void* dst,
                               hipStream_t stream) {
  const size_t pieces = packed_gate_up_bytes(is_bf16, E, I, H) / 16;
  const int block = 256;
  const size_t want = (pieces + block - 1) / block;
  const int grid = static_cast<int>(want < 65536 ? want : 65536);
  pack_gate_up_kernel<<<grid, block, 0, stream>>>(static_cast<const uint4*>(gate), static_cast<const uint4*>(up),
                                                  static_cast<uint4*>(dst), E, I, H * (is_bf16 ? 2 : 4));
  return hipGetLastError();
}

hipError_t launch_pack(const void* src, int is_bf16, int E, int N, int K, void* dst, hipStream_t stream) {
  const int rowbytes = K * (is_bf16 ? 2 : 4);
  const size_t pieces = static_cast<size_t>(E) * N * rowbytes / 16;
  const int block = 256;
  const size_t want = (pieces + block - 1) / block;
  const int grid = static_cast<int>(want < 65536 ? want : 65536);
  pack_kernel<<<grid, block, 0, stream>>>(static_cast<const uint4*>(src), static_cast<uint4*>(dst), E,
                                          N, rowbytes);
  return hipGetLastError();
}

// workspace: [cnt E | off E+1 | active E | n_active | n_items] ints, CSR slot
// ids, activations, then the per-slot output rows (row pass) or the down
// items (column-tile pass)
size_t forward_workspace_bytes(int T, int H, int I, int E, int k, int is_bf16) {
  const size_t slots = static_cast<size_t>(T) * k;
  const size_t eb = is_bf16 ? 2 : 4;
  const size_t head = align256(sizeof(int32_t) * (3 * static_cast<size_t>(E) + 3)) +
                      align256(sizeof(int32_t) * slots) + align256(slots * I * eb);
  if (use_col_path(T, k)) {
    const size_t items = (slots + 15) / 16 + (static_cast<size_t>(E) < slots ? E : slots);
    return head + align256(items * sizeof(int4));
  }
  return head + align256(slots * H * sizeof(float));
}

void forward_carve(void* ws, ForwardParams& p) {
  char* c = static_cast<char*>(ws);
  const size_t slots = static_cast<size_t>(p.T) * p.k;
  const size_t eb = p.is_bf16 ? 2 : 4;
  int32_t* ints = reinterpret_cast<int32_t*>(c);
  p.cnt = ints;
  p.off = ints + p.E;
  p.active = ints + 2 * p.E + 1;
  p.n_active = ints + 3 * p.E + 1;
  p.n_items = ints + 3 * p.E + 2;
  c += align256(sizeof(int32_t) * (3 * static_cast<size_t>(p.E) + 3));
  p.ent_slot = reinterpret_cast<int32_t*>(c);
  c += align256(sizeof(int32_t) * slots);
  p.act = c;
  c += align256(slots * p.I * eb);
  if (use_col_path(p.T, p.k)) {
    p.items = reinterpret_cast<int4*>(c);
    p.ys = nullptr;
  } else {
    p.items = nullptr;
    p.ys = reinterpret_cast<float*>(c);
  }
}

hipError_t launch_forward(ForwardParams p, hipStream_t stream) {
  const bool col = use_col_path(p.T, p.k);
  const ColShape cs = col_shape(p.T, p.H, p.I, p.is_bf16);
  p.zero_out = col && cs.ksplit == 2;
  p.item_rows = 16 * cs.mti;
  const bool small_k = p.k <= 8;
  hipError_t err = hipSuccess;
  if (!col) {
    if (small_k)
      dispatch_kernel<8><<<1, kDispatchThreads, 0, stream>>>(p);
    else
      dispatch_kernel<kMaxTopK><<<1, kDispatchThreads, 0, stream>>>(p);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  // upper bound on active experts: min(E, T*k)
  const int cap = p.E < p.T * p.k ? p.E : p.T * p.k;
  const bool small_t = p.T <= 32;
  if (p.is_bf16)
    err = small_t ? launch_gate_up<Bf16Path, 2>(p, cap, col, stream) : launch_gate_up<Bf16Path, 4>(p, cap, col, stream);
  else
    err = small_t ? launch_gate_up<F32Path, 2>(p, cap, col, stream) : launch_gate_up<F32Path, 4>(p, cap, col, stream);
  if (err != hipSuccess) return err;
  if (col) return p.is_bf16 ? launch_down_col<Bf16Path>(p, cs, stream) : launch_down_col<F32Path>(p, cs, stream);
  if (p.is_bf16)
    err = small_t ? launch_down_rows<Bf16Path, 2>(p, cap, stream) : launch_down_rows<Bf16Path, 4>(p, cap, stream);
  else
    err = small_t ? launch_down_rows<F32Path, 2>(p, cap, stream) : launch_down_rows<F32Path, 4>(p, cap, stream);
  if (err != hipSuccess) return err;
  const int hblocks = (p.H / 4 + 255) / 256;
  const dim3 cgrid(static_cast<unsigned>(hblocks) * static_cast<unsigned>(p.T));
  if (small_k)
    combine_kernel<8><<<cgrid, 256, 0, stream>>>(p, hblocks);
  else
    combine_kernel<kMaxTopK><<<cgrid, 256, 0, stream>>>(p, hblocks);
  return hipGetLastError();
}

}  // namespace amoe
