// AcceptMoE eligible-set selection, one 1024-thread workgroup per draft tree.
//
// Phases (each separated by a workgroup barrier):
//   P1  tree checks and depth counts N_d                          (Sec. 3.1, 3.2)
//   P2  per node (one wave per node): natural top-k K_t over the fp32
//       logits, r_t = softmax(z_t) in fp64, alpha_t r_{t,e} for e in K_t,
//       votes v_e and the root anchor                  (Sec. 3.1 Eq. 1, Eq. 3, Eq. 5)
//   P3  utility u_e = sum_t alpha_t r_{t,e} 1[e in K_t], summed in node order
//       through a dense LDS tile                                  (Eq. 4)
//   P4  effective rank over R = [E] \ A, self-sized set S, optional
//       residency pruning -> S'                       (Eq. 6, Sec. 3.3, Eq. 7)
//   P5  per node: restricted top-k over S' and renormalised gates  (Eq. 2)
//   P6  eligible mask and per-tree statistics
//
// Top-k is a wave-wide radix select on order-preserving 32-bit keys: the k-th
// largest key is found bit by bit with ballots, keys above it are taken,
// equal keys are taken lowest expert index first.  This matches the rank
// definition "fewer than k experts beat e" exactly, ties included.
#include "common.hpp"
#include "launch.hpp"

namespace amoe {

namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kDenseDoubles = 4096;  // P3 LDS tile: chunk_tokens * E <= this

enum { MODE_SELF = 0, MODE_ALL = 1, MODE_FIXED = 2, MODE_MOESPEC = 3, MODE_COUNT = 4 };
enum { CODE_OK = 0, CODE_EMPTY = 1, CODE_ROOT = 2, CODE_PARENT = 3, CODE_DEPTH = 4, CODE_PROB = 5 };

struct SelShared {
  int code;
  int n_anchor, n_unat, n_R, n_pos, n_S, n_C, n_Sp, n_routed;
  int n_er, n_take, budget_a, m_star;
  double Z, Hsum;
  int Nd[kMaxTreeNodes];
  int votes[kMaxExperts];
  int rankv[kMaxExperts];
  int pv[kMaxExperts];
  double u[kMaxExperts];
  double dense[kDenseDoubles];
  uint8_t anchor[kMaxExperts];
  uint8_t inS[kMaxExperts];
  uint8_t inSp[kMaxExperts];
  uint8_t routed[kMaxExperts];
  uint8_t resident[kMaxExperts];
  // per-wave compaction scratch for top-k slot ordering
  uint32_t sk[kSelWaves][kMaxTopK];
  int se[kSelWaves][kMaxTopK];
  float sz[kSelWaves][kMaxTopK];
};

// k-th largest key among the wave's EPL*64 keys (0 if fewer than k are non-zero).
template <int EPL>
__device__ __forceinline__ uint32_t kth_largest(const uint32_t (&key)[EPL], int k) {
  uint32_t cand = 0u;
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t trial = cand | (1u << bit);
    int cnt = 0;
#pragma unroll
    for (int i = 0; i < EPL; ++i) cnt += popc64(__ballot(key[i] >= trial));
    if (cnt >= k) cand = trial;
  }
  return cand;
}

// Selects the top-k keys of the wave (ties -> lower expert index) and
// compacts the winners into the wave's scratch in expert-index order.
// Returns the number selected (min(k, #non-zero keys)).
template <int EPL>
__device__ __forceinline__ int wave_topk_compact(const uint32_t (&key)[EPL], const float (&zv)[EPL],
                                                 int k, int lane, uint32_t* sk, int* se, float* sz) {
  const uint32_t thr = kth_largest<EPL>(key, k);
  int greater = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i) greater += popc64(__ballot(key[i] > thr));
  const int need = k - greater;
  const uint64_t below = lanes_below(lane);
  int eq_before = 0, base = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const bool eq = (key[i] == thr) && (key[i] != 0u);
    const uint64_t eqm = __ballot(eq);
    const bool sel = (key[i] > thr) || (eq && (eq_before + popc64(eqm & below)) < need);
    eq_before += popc64(eqm);
    const uint64_t sm = __ballot(sel);
    if (sel) {
      const int pos = base + popc64(sm & below);
      sk[pos] = key[i];
      se[pos] = lane + kWave * i;
      sz[pos] = zv[i];
    }
    base += popc64(sm);
  }
  wave_lds_sync();
  return base;
}

// Slot (rank) of compacted entry j among the n selected: (key desc, index asc).
__device__ __forceinline__ int slot_of(int j, int n, const uint32_t* sk, const int* se) {
  const uint32_t kj = sk[j];
  const int ej = se[j];
  int r = 0;
  for (int i = 0; i < n; ++i) r += (sk[i] > kj) || (sk[i] == kj && se[i] < ej);
  return r;
}

// Deterministic workgroup sum of one double per expert (E <= 512): wave 0
// adds lane-strided slices in index order, then a fixed butterfly.
__device__ __forceinline__ double wg_sum_experts(const double* vals, int E, int wave, int lane) {
  double s = 0.0;
  if (wave == 0)
    for (int e = lane; e < E; e += kWave) s += vals[e];
  return wave == 0 ? wave_sum_f64(s) : 0.0;
}

template <int EPL>
__global__ __launch_bounds__(kSelThreads) void select_kernel(SelectParams p, TreeOffsets offs) {
  __shared__ SelShared sh;
  const int tid = threadIdx.x;
  const int wave = tid / kWave, lane = lane_id();
  const int b = blockIdx.x;
  const int t_begin = offs.o[b];
  const int Tb = offs.o[b + 1] - t_begin;
  const int E = p.E, k = p.k;
  const bool has_mask = p.resident != nullptr;

  // ---------------- P1: tree checks, N_d ----------------
  if (tid == 0) {
    sh.code = Tb > 0 ? 0x7fffffff : CODE_EMPTY;
    sh.n_anchor = sh.n_unat = sh.n_R = sh.n_pos = sh.n_S = sh.n_C = sh.n_Sp = sh.n_routed = 0;
    sh.budget_a = sh.m_star = sh.n_er = sh.n_take = 0;
  }
  for (int i = tid; i < kMaxTreeNodes; i += kSelThreads) sh.Nd[i] = 0;
  for (int e = tid; e < E; e += kSelThreads) {
    sh.votes[e] = 0;
    sh.anchor[e] = 0;
    sh.inS[e] = 0;
    sh.inSp[e] = 0;
    sh.routed[e] = 0;
    sh.resident[e] = has_mask ? (p.resident[e] != 0) : 1;
  }
  __syncthreads();
  for (int tl = tid; tl < Tb; tl += kSelThreads) {
    const int t = t_begin + tl;
    const int d = p.depth[t];
    int code = 0;
    if (tl == 0) {
      if (d != 0 || (p.parent != nullptr && p.parent[t] != -1)) code = CODE_ROOT;
    } else if (p.parent != nullptr) {
      const int par = p.parent[t];
      if (par < t_begin || par >= t) code = CODE_PARENT;
      else if (d != p.depth[par] + 1) code = CODE_DEPTH;
    } else if (d < 1 || d >= Tb) {
      code = CODE_DEPTH;
    }
    const float pr = p.prob[t];
    if (!(pr >= 0.0f) || !isfinite(pr)) code = code ? code : CODE_PROB;
    if (code) atomicMin(&sh.code, code);
    if (d >= 0 && d < Tb) atomicAdd(&sh.Nd[d], 1);
  }
  __syncthreads();
  const int code = (sh.code == 0x7fffffff) ? 0 : sh.code;

  if (code != 0) {
    // invalid tree: no routing for its nodes
    for (int i = tid; i < Tb * k; i += kSelThreads) {
      p.topk_idx[static_cast<size_t>(t_begin) * k + i] = -1;
      p.topk_gate[static_cast<size_t>(t_begin) * k + i] = 0.0f;
    }
    for (int e = tid; e < E; e += kSelThreads) p.eligible[static_cast<size_t>(b) * E + e] = 0;
    if (p.stats != nullptr && tid < kNumStats) {
      int v = 0;
      if (tid == 0) v = Tb;
      if (tid == 8) v = code;
      p.stats[b * kNumStats + tid] = v;
    }
    return;
  }

  // ---------------- P2: natural top-k, softmax, contributions ----------------
  uint32_t* sk = sh.sk[wave];
  int* se = sh.se[wave];
  float* sz = sh.sz[wave];
  for (int tl = wave; tl < Tb; tl += kSelWaves) {
    const int t = t_begin + tl;
    const float* zrow = p.logits + static_cast<size_t>(t) * E;
    float zv[EPL];
    uint32_t key[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = lane + kWave * i;
      zv[i] = e < E ? zrow[e] : -INFINITY;
      key[i] = e < E ? logit_key(zv[i]) : 0u;
    }
    // softmax over all E in fp64 (max subtracted)
    float zmax = zv[0];
#pragma unroll
    for (int i = 1; i < EPL; ++i) zmax = fmaxf(zmax, zv[i]);
    zmax = wave_max_f32(zmax);
    double den = 0.0;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (lane + kWave * i < E) den += exp(static_cast<double>(zv[i]) - static_cast<double>(zmax));
    den = wave_sum_f64(den);
    if (p.mode == MODE_MOESPEC) {
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        const int e = lane + kWave * i;
        if (e < E)
          p.ws_rfull[static_cast<size_t>(t) * E + e] =
              exp(static_cast<double>(zv[i]) - static_cast<double>(zmax)) / den;
      }
    }
    const int d = p.depth[t];
    const double alpha = pow(static_cast<double>(p.prob[t]), p.beta) / sqrt(static_cast<double>(sh.Nd[d]));
    const int n = wave_topk_compact<EPL>(key, zv, k, lane, sk, se, sz);
    if (lane < n) {
      const int slot = slot_of(lane, n, sk, se);
      const int e = se[lane];
      const double r = exp(static_cast<double>(sz[lane]) - static_cast<double>(zmax)) / den;
      p.ws_kidx[static_cast<size_t>(t) * k + slot] = e;
      p.ws_contrib[static_cast<size_t>(t) * k + slot] = alpha * r;
      atomicAdd(&sh.votes[e], 1);
      if (d == 0) sh.anchor[e] = 1;
    }
    wave_lds_sync();
  }
  __syncthreads();

  // ---------------- P3: utility in node order ----------------
  double u_acc = 0.0;
  const int chunk = kDenseDoubles / E;  // >= 8 for E <= 512
  for (int c0 = 0; c0 < Tb; c0 += chunk) {
    const int cn = min(chunk, Tb - c0);
    for (int i = tid; i < cn * E; i += kSelThreads) sh.dense[i] = 0.0;
    __syncthreads();
    for (int i = tid; i < cn * k; i += kSelThreads) {
      const int tl = c0 + i / k;
      const size_t gi = static_cast<size_t>(t_begin + tl) * k + (i % k);
      const int e = p.ws_kidx[gi];
      sh.dense[(tl - c0) * E + e] = p.ws_contrib[gi];
    }
    __syncthreads();
    if (tid < E)
      for (int j = 0; j < cn; ++j) u_acc += sh.dense[j * E + tid];
    __syncthreads();
  }
  if (tid < E) sh.u[tid] = u_acc;
  __syncthreads();

  // ---------------- P4: eligible set ----------------
  // counts: |A|, |U_nat|, |R|, #positive residual
  if (tid < E) {
    if (sh.anchor[tid]) atomicAdd(&sh.n_anchor, 1);
    if (sh.votes[tid] > 0) atomicAdd(&sh.n_unat, 1);
    if (!sh.anchor[tid]) {
      atomicAdd(&sh.n_R, 1);
      if (sh.u[tid] > 0.0) atomicAdd(&sh.n_pos, 1);
    }
  }
  __syncthreads();
  const int mode = p.mode;
  const int kmin = min(k, E);
  int bud = p.budget < kmin ? kmin : (p.budget > E ? E : p.budget);

  if (mode == MODE_SELF) {
    // Z = sum over R of u^+ ; H = -sum q log q ; n_er = ceil(exp(H) - 1e-9)
    if (tid < E) sh.dense[tid] = (!sh.anchor[tid] && sh.u[tid] > 0.0) ? sh.u[tid] : 0.0;
    __syncthreads();
    const double Z = wg_sum_experts(sh.dense, E, wave, lane);
    if (tid == 0) sh.Z = Z;
    __syncthreads();
    const double Zs = sh.Z;
    if (tid < E) {
      const double uu = sh.dense[tid];
      double term = 0.0;
      if (uu > 0.0 && Zs > 0.0) {
        const double q = uu / Zs;
        term = q * log(q);
      }
      sh.dense[kMaxExperts + tid] = term;
    }
    __syncthreads();
    const double hs = wg_sum_experts(sh.dense + kMaxExperts, E, wave, lane);
    if (tid == 0) {
      int ner = 0;
      if (Zs > 0.0) {
        const double x = exp(-hs);
        ner = static_cast<int>(ceil(x - 1e-9));
        if (ner < 1) ner = 1;
        if (ner > sh.n_pos) ner = sh.n_pos;
      }
      sh.n_er = ner;
      int take = ner;
      if (sh.n_anchor + take < kmin) take = kmin - sh.n_anchor;
      if (take > sh.n_R) take = sh.n_R;
      sh.n_take = take;
    }
  } else if (mode == MODE_FIXED) {
    if (tid == 0) {
      int take = bud - sh.n_anchor;
      if (take < 0) take = 0;
      if (take > sh.n_R) take = sh.n_R;
      sh.n_er = take;
      sh.n_take = take;
    }
  }
  __syncthreads();

  if (mode == MODE_SELF || mode == MODE_FIXED) {
    // rank within R by (u desc, index asc); S = A u first n_take of R
    if (tid < E) {
      bool in = sh.anchor[tid] != 0;
      if (!in) {
        const double ue = sh.u[tid];
        int r = 0;
        for (int j = 0; j < E; ++j)
          if (!sh.anchor[j]) {
            const double uj = sh.u[j];
            r += (uj > ue) || (uj == ue && j < tid);
          }
        in = r < sh.n_take;
      }
      sh.inS[tid] = in;
    }
  } else if (mode == MODE_ALL) {
    if (tid < E) sh.inS[tid] = 1;
  } else {
    // MoE-Spec (summed router mass) or Count-B (votes): top-bud of all experts
    double score = 0.0;
    if (tid < E) {
      if (mode == MODE_MOESPEC) {
        for (int tl = 0; tl < Tb; ++tl) score += p.ws_rfull[static_cast<size_t>(t_begin + tl) * E + tid];
      } else {
        score = static_cast<double>(sh.votes[tid]);
      }
      sh.dense[tid] = score;
    }
    __syncthreads();
    if (tid < E) {
      int r = 0;
      for (int j = 0; j < E; ++j) {
        const double sj = sh.dense[j];
        r += (sj > score) || (sj == score && j < tid);
      }
      sh.inS[tid] = r < bud;
    }
  }
  __syncthreads();

  // |S|, a(S)
  if (tid < E) {
    if (sh.inS[tid]) atomicAdd(&sh.n_S, 1);
    if (!sh.inS[tid] && sh.votes[tid] > 0) atomicAdd(&sh.budget_a, sh.votes[tid]);
  }
  __syncthreads();
  if (mode == MODE_ALL) {
    if (tid == 0) {
      sh.n_er = E - sh.n_anchor;
      sh.budget_a = 0;
    }
  } else if (mode == MODE_MOESPEC || mode == MODE_COUNT) {
    // members outside the anchor
    if (tid < E && sh.inS[tid] && !sh.anchor[tid]) atomicAdd(&sh.n_er, 1);
  }

  const bool prune = has_mask && (mode == MODE_SELF || mode == MODE_FIXED);
  if (prune) {
    // C = nonresident members of S ordered by (u asc, index asc)
    if (tid < E) {
      const bool inC = sh.inS[tid] && !sh.resident[tid];
      sh.rankv[tid] = -1;
      if (inC) {
        atomicAdd(&sh.n_C, 1);
        const double ue = sh.u[tid];
        int r = 0;
        for (int j = 0; j < E; ++j)
          if (sh.inS[j] && !sh.resident[j]) {
            const double uj = sh.u[j];
            r += (uj < ue) || (uj == ue && j < tid);
          }
        sh.rankv[tid] = r;
        sh.pv[r] = sh.votes[tid];
      }
    }
    __syncthreads();
    if (tid == 0) {
      int cap = p.removal_cap < 0 ? E : p.removal_cap;
      int limit = sh.n_C;
      if (sh.n_S - k < limit) limit = sh.n_S - k;
      if (cap < limit) limit = cap;
      if (limit < 0) limit = 0;
      int m = 0, acc = 0;
      while (m < limit && acc + sh.pv[m] <= sh.budget_a) {
        acc += sh.pv[m];
        ++m;
      }
      sh.m_star = m;
    }
    __syncthreads();
    if (tid < E) sh.inSp[tid] = sh.inS[tid] && !(sh.rankv[tid] >= 0 && sh.rankv[tid] < sh.m_star);
  } else {
    if (tid < E) sh.inSp[tid] = sh.inS[tid];
  }
  __syncthreads();
  if (tid < E && sh.inSp[tid]) atomicAdd(&sh.n_Sp, 1);

  // ---------------- P5: restricted top-k and gates ----------------
  for (int tl = wave; tl < Tb; tl += kSelWaves) {
    const int t = t_begin + tl;
    const float* zrow = p.logits + static_cast<size_t>(t) * E;
    float zv[EPL];
    uint32_t key[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = lane + kWave * i;
      const bool ok = e < E && sh.inSp[e];
      zv[i] = ok ? zrow[e] : -INFINITY;
      key[i] = ok ? logit_key(zv[i]) : 0u;
    }
    const int n = wave_topk_compact<EPL>(key, zv, k, lane, sk, se, sz);
    // gates: softmax over the selected logits, fp64
    double zm = lane < n ? static_cast<double>(sz[lane]) : -INFINITY;
    zm = wave_max_f64(zm);
    const double w = lane < n ? exp(static_cast<double>(sz[lane]) - zm) : 0.0;
    const double ws = wave_sum_f64(w);
    int32_t* orow = p.topk_idx + static_cast<size_t>(t) * k;
    float* grow = p.topk_gate + static_cast<size_t>(t) * k;
    if (lane < n) {
      const int slot = slot_of(lane, n, sk, se);
      orow[slot] = se[lane];
      grow[slot] = static_cast<float>(w / ws);
      sh.routed[se[lane]] = 1;
    } else if (lane < k) {
      orow[lane] = -1;  // fewer eligible experts than k (cannot happen when |S'| >= k)
      grow[lane] = 0.0f;
    }
    wave_lds_sync();
  }
  __syncthreads();

  // ---------------- P6: outputs ----------------
  if (tid < E) {
    p.eligible[static_cast<size_t>(b) * E + tid] = sh.inSp[tid];
    if (sh.routed[tid]) atomicAdd(&sh.n_routed, 1);
  }
  __syncthreads();
  if (p.stats != nullptr && tid == 0) {
    int32_t* st = p.stats + b * kNumStats;
    st[0] = Tb;
    st[1] = sh.n_anchor;
    st[2] = sh.n_er;
    st[3] = sh.n_S;
    st[4] = sh.n_Sp;
    st[5] = sh.n_unat;
    st[6] = sh.budget_a;
    st[7] = sh.m_star;
    st[8] = 0;
    st[9] = sh.n_routed;
  }
}

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

}  // namespace

size_t select_workspace_bytes(int T, int E, int k) {
  const size_t Tt = static_cast<size_t>(T > 0 ? T : 0);
  return align256(Tt * k * sizeof(int32_t)) + align256(Tt * k * sizeof(double)) +
         align256(Tt * E * sizeof(double));
}

void select_carve(void* ws, int T, int E, int k, SelectParams& p) {
  char* c = static_cast<char*>(ws);
  const size_t Tt = static_cast<size_t>(T > 0 ? T : 0);
  p.ws_kidx = reinterpret_cast<int32_t*>(c);
  c += align256(Tt * k * sizeof(int32_t));
  p.ws_contrib = reinterpret_cast<double*>(c);
  c += align256(Tt * k * sizeof(double));
  p.ws_rfull = reinterpret_cast<double*>(c);
}

hipError_t launch_select(const SelectParams& p, const TreeOffsets& offs, hipStream_t stream) {
  const int epl = (p.E + kWave - 1) / kWave;
  dim3 grid(p.B), block(kSelThreads);
  if (epl <= 1)
    select_kernel<1><<<grid, block, 0, stream>>>(p, offs);
  else if (epl <= 2)
    select_kernel<2><<<grid, block, 0, stream>>>(p, offs);
  else if (epl <= 4)
    select_kernel<4><<<grid, block, 0, stream>>>(p, offs);
  else
    select_kernel<8><<<grid, block, 0, stream>>>(p, offs);
  return hipGetLastError();
}

}  // namespace amoe
