// Grouped SwiGLU expert FFN over the restricted routing (Sec. 3.1, Eq. 2):
// only experts that receive a token are streamed, each exactly once.
//
//   dispatch   one workgroup: per-expert token lists in node order (CSR) and
//              the list of active experts
//   gate_up    per (active expert, 16-row tile of I): X_e W_g^T and X_e W_u^T on
//              MFMA (tokens on the 16-wide M side), SwiGLU in registers, the
//              activation written once
//   down       per (active expert, 16-row tile of H): act_e W_d^T, scaled by
//              the gate and written to the token's slot row
//   combine    out_t = sum over the k slots of token t, in slot order
//
// Weights are read in the packed fragment layout (see
// acceptmoe_pack_expert_weights): one wave load = one contiguous 1 KiB block.
#include "common.hpp"
#include "launch.hpp"

namespace amoe {

namespace {

constexpr int kDispatchThreads = 1024;
constexpr int kDispatchChunk = 512;   // tokens per bitmask pass (32 KiB of LDS masks)

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

// Expert served by slot s = t*k + j, or -1 when the slot takes no part in the
// dispatch: the index lies outside [0, E), or repeats an expert of an earlier
// slot of the same token (a repeated expert is used once, at its first slot).
__device__ __forceinline__ int slot_expert(const int32_t* __restrict__ idx, int s, int k, int E) {
  const int e = idx[s];
  if (e < 0 || e >= E) return -1;
  for (int j = (s / k) * k; j < s; ++j)
    if (idx[j] == e) return -1;
  return e;
}

// ---------------------------------------------------------------------------
// dispatch: CSR of (expert -> slot ids in node order), active expert list
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kDispatchThreads) void dispatch_kernel(ForwardParams p) {
  __shared__ int s_cnt[kMaxExperts];
  __shared__ int s_off[kMaxExperts + 1];
  __shared__ int s_run[kMaxExperts];
  __shared__ uint32_t s_mask[kMaxExperts * (kDispatchChunk / 32)];
  __shared__ int s_nact;
  const int tid = threadIdx.x;
  const int E = p.E, k = p.k, T = p.T;
  const int nslot = T * k;
  for (int e = tid; e < E; e += kDispatchThreads) {
    s_cnt[e] = 0;
    s_run[e] = 0;
  }
  __syncthreads();
  for (int s = tid; s < nslot; s += kDispatchThreads) {
    const int e = slot_expert(p.topk_idx, s, k, E);
    if (e >= 0) atomicAdd(&s_cnt[e], 1);
  }
  __syncthreads();
  if (tid < kWave) {
    // exclusive scan over experts and compaction of active ones, in index order
    int base = 0, abase = 0;
    for (int e0 = 0; e0 < E; e0 += kWave) {
      const int e = e0 + tid;
      const int c = e < E ? s_cnt[e] : 0;
      int incl = c;
      for (int o = 1; o < kWave; o <<= 1) {
        const int v = __shfl_up(incl, o, kWave);
        if (tid >= o) incl += v;
      }
      if (e < E) s_off[e] = base + incl - c;
      const uint64_t am = __ballot(c > 0);
      if (c > 0) p.active[abase + popc64(am & lanes_below(tid))] = e;
      abase += popc64(am);
      base += __shfl(incl, kWave - 1, kWave);
    }
    if (tid == 0) {
      s_off[E] = base;
      s_nact = abase;
      *p.n_active = abase;
    }
  }
  __syncthreads();
  for (int e = tid; e < E; e += kDispatchThreads) {
    p.cnt[e] = s_cnt[e];
    p.off[e] = s_off[e];
  }
  if (tid == 0) p.off[E] = s_off[E];
  // position of each slot inside its expert list = earlier tokens of that expert
  const int words = kDispatchChunk / 32;
  for (int t0 = 0; t0 < T; t0 += kDispatchChunk) {
    const int tn = min(kDispatchChunk, T - t0);
    for (int i = tid; i < E * words; i += kDispatchThreads) s_mask[i] = 0u;
    __syncthreads();
    for (int i = tid; i < tn * k; i += kDispatchThreads) {
      const int tl = i / k;
      const int e = slot_expert(p.topk_idx, (t0 + tl) * k + (i % k), k, E);
      if (e >= 0) atomicOr(&s_mask[e * words + (tl >> 5)], 1u << (tl & 31));
    }
    __syncthreads();
    for (int i = tid; i < tn * k; i += kDispatchThreads) {
      const int tl = i / k;
      const int s = (t0 + tl) * k + (i % k);
      const int e = slot_expert(p.topk_idx, s, k, E);
      if (e >= 0) {
        const uint32_t* m = s_mask + e * words;
        int before = 0;
        for (int w = 0; w < (tl >> 5); ++w) before += __popc(m[w]);
        before += __popc(m[tl >> 5] & ((1u << (tl & 31)) - 1u));
        p.ent_slot[s_off[e] + s_run[e] + before] = s;
      }
    }
    __syncthreads();
    for (int e = tid; e < E; e += kDispatchThreads) {
      int c = 0;
      for (int w = 0; w < words; ++w) c += __popc(s_mask[e * words + w]);
      s_run[e] += c;
    }
    __syncthreads();
  }
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

// ---------------------------------------------------------------------------
// gate/up + SwiGLU.  grid.x = cap_experts * ceil(NT/4), block 256: wave w of
// workgroup (a, q) owns I-tile nt = 4q + w of active expert a.
// ---------------------------------------------------------------------------
template <class P, int MT>
__global__ __launch_bounds__(256) void gateup_kernel(ForwardParams p) {
  const int NT = p.I / 16;
  const int wg_per_expert = (NT + 3) / 4;
  const int a = blockIdx.x / wg_per_expert;
  const int nt = (blockIdx.x % wg_per_expert) * 4 + threadIdx.x / kWave;
  if (a >= *p.n_active || nt >= NT) return;
  const int lane = lane_id();
  const int r = lane & 15, g = lane >> 4;
  const int e = p.active[a];
  const int n_e = p.cnt[e];
  const int o_e = p.off[e];
  const int H = p.H, I = p.I;
  const int KC = H / P::kKF;                 // fragments along K
  const int rowq = H * P::kElemBytes / 16;   // 16-B pieces per hidden row

  const uint4* hid = static_cast<const uint4*>(p.hidden);
  const size_t frag0 = (static_cast<size_t>(e) * NT + nt) * KC;
  const uint4* bg = static_cast<const uint4*>(p.w_gate) + frag0 * kWave + lane;
  const uint4* bu = static_cast<const uint4*>(p.w_up) + frag0 * kWave + lane;

  for (int m0 = 0; m0 < n_e; m0 += 16 * MT) {
    const int nmt = min(MT, (n_e - m0 + 15) / 16);
    const uint4* ap[MT];
    bool av[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = m0 + mt * 16 + r;
      av[mt] = (mt < nmt) && (m < n_e);
      const int tok = av[mt] ? p.ent_slot[o_e + m] / p.k : 0;
      ap[mt] = hid + static_cast<size_t>(tok) * rowq + g;
    }
    floatx4 accg[MT], accu[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      accg[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
      accu[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll 4
    for (int kc = 0; kc < KC; ++kc) {
      const uint4 wg = bg[static_cast<size_t>(kc) * kWave];
      const uint4 wu = bu[static_cast<size_t>(kc) * kWave];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        if (mt < nmt) {
          const uint4 x = av[mt] ? ap[mt][kc * 4] : make_uint4(0u, 0u, 0u, 0u);
          accg[mt] = P::mma(x, wg, accg[mt]);
          accu[mt] = P::mma(x, wu, accu[mt]);
        }
      }
    }
    // epilogue: act[o_e + m][nt*16 + r] for rows m = m0 + mt*16 + 4g + i
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      if (mt >= nmt) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + mt * 16 + 4 * g + i;
        if (m < n_e) {
          const float v = silu_mul(accg[mt][i], accu[mt][i]);
          const size_t idx = static_cast<size_t>(o_e + m) * I + nt * 16 + r;
          if (P::kElemBytes == 2)
            static_cast<uint16_t*>(p.act)[idx] = float_to_bf16_bits(v);
          else
            static_cast<float*>(p.act)[idx] = v;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// down projection.  grid.x = cap_experts * ceil(HT/4); wave w of workgroup
// (a, q) owns H-tile ht = 4q + w of active expert a.
// ---------------------------------------------------------------------------
template <class P, int MT>
__global__ __launch_bounds__(256) void down_kernel(ForwardParams p) {
  const int HT = p.H / 16;
  const int wg_per_expert = (HT + 3) / 4;
  const int a = blockIdx.x / wg_per_expert;
  const int ht = (blockIdx.x % wg_per_expert) * 4 + threadIdx.x / kWave;
  if (a >= *p.n_active || ht >= HT) return;
  const int lane = lane_id();
  const int r = lane & 15, g = lane >> 4;
  const int e = p.active[a];
  const int n_e = p.cnt[e];
  const int o_e = p.off[e];
  const int H = p.H, I = p.I;
  const int KC = I / P::kKF;
  const int rowq = I * P::kElemBytes / 16;

  const uint4* act = static_cast<const uint4*>(p.act);
  const size_t frag0 = (static_cast<size_t>(e) * HT + ht) * KC;
  const uint4* bd = static_cast<const uint4*>(p.w_down) + frag0 * kWave + lane;

  for (int m0 = 0; m0 < n_e; m0 += 16 * MT) {
    const int nmt = min(MT, (n_e - m0 + 15) / 16);
    const uint4* ap[MT];
    bool av[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int m = m0 + mt * 16 + r;
      av[mt] = (mt < nmt) && (m < n_e);
      ap[mt] = act + static_cast<size_t>(av[mt] ? o_e + m : 0) * rowq + g;
    }
    floatx4 acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
    for (int kc = 0; kc < KC; ++kc) {
      const uint4 w = bd[static_cast<size_t>(kc) * kWave];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        if (mt < nmt) {
          const uint4 x = av[mt] ? ap[mt][kc * 4] : make_uint4(0u, 0u, 0u, 0u);
          acc[mt] = P::mma(x, w, acc[mt]);
        }
      }
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      if (mt >= nmt) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + mt * 16 + 4 * g + i;
        if (m < n_e) {
          const int s = p.ent_slot[o_e + m];
          p.ys[static_cast<size_t>(s) * H + ht * 16 + r] = p.topk_gate[s] * acc[mt][i];
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// combine: out[t, h] = sum_j ys[t*k + j, h] over valid slots, slot order
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void combine_kernel(ForwardParams p) {
  const int t = blockIdx.y;
  const int h4 = blockIdx.x * blockDim.x + threadIdx.x;  // float4 column
  const int H = p.H, k = p.k;
  if (h4 * 4 >= H) return;
  float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int j = 0; j < k; ++j) {
    if (slot_expert(p.topk_idx, t * k + j, k, p.E) < 0) continue;
    const float4 v = reinterpret_cast<const float4*>(p.ys + static_cast<size_t>(t * k + j) * H)[h4];
    s.x += v.x;
    s.y += v.y;
    s.z += v.z;
    s.w += v.w;
  }
  reinterpret_cast<float4*>(p.out + static_cast<size_t>(t) * H)[h4] = s;
}

template <class P, int MT>
hipError_t launch_ffn(const ForwardParams& p, int cap, hipStream_t stream) {
  const int gu_wg = (p.I / 16 + 3) / 4;
  const int dn_wg = (p.H / 16 + 3) / 4;
  gateup_kernel<P, MT><<<dim3(cap * gu_wg), 256, 0, stream>>>(p);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  down_kernel<P, MT><<<dim3(cap * dn_wg), 256, 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace

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

size_t forward_workspace_bytes(int T, int H, int I, int E, int k, int is_bf16) {
  const size_t slots = static_cast<size_t>(T) * k;
  const size_t eb = is_bf16 ? 2 : 4;
  return align256(sizeof(int32_t) * (3 * static_cast<size_t>(E) + 2)) + align256(sizeof(int32_t) * slots) +
         align256(slots * I * eb) + align256(slots * H * sizeof(float));
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
  c += align256(sizeof(int32_t) * (3 * static_cast<size_t>(p.E) + 2));
  p.ent_slot = reinterpret_cast<int32_t*>(c);
  c += align256(sizeof(int32_t) * slots);
  p.act = c;
  c += align256(slots * p.I * eb);
  p.ys = reinterpret_cast<float*>(c);
}

hipError_t launch_forward(const ForwardParams& p, hipStream_t stream) {
  dispatch_kernel<<<1, kDispatchThreads, 0, stream>>>(p);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  // upper bound on active experts: min(E, T*k)
  const int cap = p.E < p.T * p.k ? p.E : p.T * p.k;
  if (p.is_bf16) {
    err = p.T <= 32 ? launch_ffn<Bf16Path, 2>(p, cap, stream) : launch_ffn<Bf16Path, 4>(p, cap, stream);
  } else {
    err = p.T <= 32 ? launch_ffn<F32Path, 2>(p, cap, stream) : launch_ffn<F32Path, 4>(p, cap, stream);
  }
  if (err != hipSuccess) return err;
  dim3 cgrid((p.H / 4 + 255) / 256, p.T);
  combine_kernel<<<cgrid, 256, 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace amoe
