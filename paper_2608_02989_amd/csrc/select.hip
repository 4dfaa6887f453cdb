// AcceptMoE eligible-set selection.
//
//   natural top-k     per node: K_t over the fp32 logits and r_t = softmax(z_t)
//                     in fp64 for the selected experts           (Sec. 3.1, Eq. 1)
//   tree stage        per draft tree:
//     P1  depth / parent / probability of every node; tree checks, depth
//         counts N_d, importance alpha_t = p_t^beta / sqrt(N_{d_t})   (Eq. 3)
//     P3  utility u_e = sum_t alpha_t r_{t,e} 1[e in K_t], summed in node order
//         through a dense LDS tile; votes v_e; root anchor A         (Eq. 4, Eq. 5)
//     P4  effective rank over R = [E] \ A, self-sized set S, optional
//         residency pruning -> S'                        (Eq. 6, Sec. 3.3, Eq. 7)
//   restricted top-k  per node: top-k over S' and renormalised gates   (Eq. 2)
//
// Three launches: natural_kernel and restricted_kernel put one wave on each
// node and spread the nodes over many CUs; tree_kernel runs one 1024-thread
// workgroup per tree between them.  The per-node top-k is bound by
// instruction issue (a ballot search over the key bits, fp64 exponentials):
// a block's nodes on one CU queue behind each other on its four SIMDs, which
// costs more than the two launches saved by running everything in one
// workgroup.
//
// Top-k is a wave-wide radix select on order-preserving keys: the k-th
// largest key is found bit by bit with ballots (stopping once exactly k keys
// remain above the prefix), keys above it are taken, equal keys are taken
// lowest expert index first.  This matches the rank definition "fewer than k
// experts beat e" exactly, ties included.
#include <mutex>

#include "abi_util.hpp"
#include "common.hpp"
#include "launch.hpp"

namespace amoe {

namespace {

constexpr int kSelThreads = 1024;
constexpr int kNodeWaves = 4;        // nodes per workgroup in the per-node kernels
// P3 LDS tile: chunk_tokens * E <= this.  64 nodes at E = 128 fit in one
// chunk (one barrier pair instead of two; the sums run in node order either
// way, so the result does not depend on the chunk size): the 48-layer pass at
// T = 60 ran 4956 -> 4925 us per block with 8192 instead of 4096 doubles.
constexpr int kDenseDoubles = 8192;
constexpr int kRoutedWords = kMaxExperts / 32;

enum { MODE_SELF = 0, MODE_ALL = 1, MODE_FIXED = 2, MODE_MOESPEC = 3, MODE_COUNT = 4 };
enum { CODE_OK = 0, CODE_EMPTY = 1, CODE_ROOT = 2, CODE_PARENT = 3, CODE_DEPTH = 4, CODE_PROB = 5 };

struct SelShared {
  int code;
  int n_anchor, n_unat, n_R, n_pos, n_S, n_C, n_Sp, n_routed;
  int n_er, n_take, budget_a, m_star;
  alignas(16) int Nd[kMaxTreeNodes];
  alignas(16) double alpha[kMaxTreeNodes];
  alignas(16) int votes[kMaxExperts];
  alignas(16) int rankv[kMaxExperts];
  alignas(16) int pv[kMaxExperts];
  alignas(16) double u[kMaxExperts];
  alignas(16) double score[kMaxExperts];
  alignas(16) double dense[kDenseDoubles];
  // per-expert flags (entries E..kMaxExperts-1 stay 0)
  alignas(16) uint8_t anchor[kMaxExperts];
  alignas(16) uint8_t inR[kMaxExperts];
  alignas(16) uint8_t inS[kMaxExperts];
  alignas(16) uint8_t inC[kMaxExperts];
  alignas(16) uint8_t inSp[kMaxExperts];
  alignas(16) uint8_t routed[kMaxExperts];
  alignas(16) uint8_t resident[kMaxExperts];
  alignas(16) int rpart[kSelThreads];  // partial rank counts
  alignas(16) int plist[kMaxExperts];     // compacted expert lists (positive R members, then C) ...
  alignas(16) double pval[kMaxExperts];   // ... and their utilities
};

// compaction scratch of one node's top-k (slot ordering)
struct NodeSlot {
  alignas(16) uint32_t sk[kMaxTopK];
  alignas(16) int se[kMaxTopK];
  alignas(16) float sz[kMaxTopK];
  alignas(16) double sx[kMaxTopK];
};
struct NodeScratch {
  NodeSlot s[kNodeWaves];
};

// Wave minimum of 32-bit keys, broadcast (the DPP steps of dpp::reduce).
__device__ __forceinline__ uint32_t wave_min_key(uint32_t v) {
  return dpp::reduce(v, 0xffffffffu, [](uint32_t x, uint32_t y) { return min(x, y); });
}

// k-th largest key among the wave's EPL*64 32-bit keys, for NN
// nodes at once (0 if fewer than k keys are non-zero).  The key is built from
// the top bit down: cand grows while at least k keys stay >= cand.  Once
// exactly k keys are >= cand that count stays k, those keys are the top k and
// the answer is their smallest, so the search stops at the next check (for
// logits usually after a third of the bits) and takes that minimum; the
// result equals the full search.  Bits go in unrolled groups of four with one
// check per group (a wave issues one instruction at a time: a check per bit
// would double the cost of a step).  The NN searches are independent; one
// loop lets their ballot chains interleave.
template <int EPL, int NN, class Key>
__device__ __forceinline__ void kth_largest(const Key (&key)[NN][EPL], int k, Key (&cand)[NN]) {
  constexpr int kBits = 8 * sizeof(Key);
  int have[NN];  // number of keys >= cand[j]
#pragma unroll
  for (int j = 0; j < NN; ++j) {
    cand[j] = 0;
    have[j] = EPL * kWave;
  }
  for (int b0 = kBits - 1; b0 >= 0; b0 -= 4) {
    bool open = false;
#pragma unroll
    for (int j = 0; j < NN; ++j) open = open || have[j] != k;
    if (!open) break;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
#pragma unroll
      for (int j = 0; j < NN; ++j) {
        const Key trial = cand[j] | (static_cast<Key>(1) << (b0 - d));
        int cnt = 0;
#pragma unroll
        for (int i = 0; i < EPL; ++i) cnt += popc64(__ballot(key[j][i] >= trial));
        if (cnt >= k) {
          cand[j] = trial;
          have[j] = cnt;
        }
      }
    }
  }
#pragma unroll
  for (int j = 0; j < NN; ++j) {
    if (have[j] != k) continue;  // the search ran to the last bit: cand is exact
    Key m = ~static_cast<Key>(0);
#pragma unroll
    for (int i = 0; i < EPL; ++i) m = key[j][i] >= cand[j] ? min(m, key[j][i]) : m;
    cand[j] = wave_min_key(m);
  }
}

// Takes the top-k keys of the wave given their threshold thr = k-th largest
// key (ties -> lower expert index) and compacts the winners into the node's
// scratch in expert-index order: key and expert index, plus put(pos, i) for
// the caller's own payload of element i.  Returns the number selected
// (min(k, #non-zero keys)).
template <int EPL, class Put>
__device__ __forceinline__ int topk_compact(uint32_t thr, const uint32_t (&key)[EPL], int k, int lane, uint32_t* sk,
                                            int* se, Put&& put) {
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
    const bool sel = (key[i] > thr) | (eq & ((eq_before + popc64(eqm & below)) < need));
    eq_before += popc64(eqm);
    const uint64_t sm = __ballot(sel);
    if (sel) {
      const int pos = base + popc64(sm & below);
      sk[pos] = key[i];
      se[pos] = lane + kWave * i;
      put(pos, i);
    }
    base += popc64(sm);
  }
  wave_lds_sync();
  return base;
}

// Slot (rank) of compacted entry j among the n selected: (key desc, index asc).
// Reads the scratch four entries at a time.
__device__ __forceinline__ int slot_of(int j, int n, const uint32_t* sk, const int* se) {
  const uint32_t kj = sk[j];
  const int ej = se[j];
  int r = 0;
  for (int i0 = 0; i0 < n; i0 += 4) {
    const uint4 kk = *reinterpret_cast<const uint4*>(sk + i0);
    const int4 ee = *reinterpret_cast<const int4*>(se + i0);
    // bitwise (not short-circuit) logic keeps this branch-free
    r += static_cast<int>((i0 + 0 < n) & ((kk.x > kj) | ((kk.x == kj) & (ee.x < ej))));
    r += static_cast<int>((i0 + 1 < n) & ((kk.y > kj) | ((kk.y == kj) & (ee.y < ej))));
    r += static_cast<int>((i0 + 2 < n) & ((kk.z > kj) | ((kk.z == kj) & (ee.z < ej))));
    r += static_cast<int>((i0 + 3 < n) & ((kk.w > kj) | ((kk.w == kj) & (ee.w < ej))));
  }
  return r;
}

// rank[e] for every flagged e (0 for unflagged experts): the E x E comparison
// is split over all threads of the workgroup, thread (part, e) counting the
// flagged competitors of e in one slice of the index range (threads of a wave
// share the slice, so their LDS reads are broadcasts); the partial counts are
// stored and added per expert after a barrier.  The caller synchronizes
// before reading rank.
// slices of the index range per expert in rank_item (E * parts <= kSelThreads)
__device__ __forceinline__ int rank_parts(int E) { return E <= 128 ? 8 : (E <= 256 ? 4 : 2); }

// Partial rank of flagged expert e (item = part * E + e): the flagged
// competitors in index slice `part` that come before e in (v desc or asc,
// index asc) order; 0 for an unflagged e.  Eight broadcast values per LDS
// step (flags past E are 0, reads stay inside the kMaxExperts arrays).
template <bool kDesc>
__device__ __forceinline__ int rank_item(const double* v, const uint8_t* flag, int E, int parts, int item) {
  const int span = ((E + parts - 1) / parts + 7) & ~7;  // competitors per slice, multiple of 8
  const int part = item / E, e = item % E;
  const double ve = v[e];
  const int j_begin = part * span;
  const int j_end = min(E, j_begin + span);
  int r = 0;
  for (int j0 = j_begin; j0 < j_end; j0 += 8) {
    const double2 a = *reinterpret_cast<const double2*>(v + j0);
    const double2 b = *reinterpret_cast<const double2*>(v + j0 + 2);
    const double2 c = *reinterpret_cast<const double2*>(v + j0 + 4);
    const double2 d = *reinterpret_cast<const double2*>(v + j0 + 6);
    const uint2 f = *reinterpret_cast<const uint2*>(flag + j0);
    const double vv[8] = {a.x, a.y, b.x, b.y, c.x, c.y, d.x, d.y};
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const bool fl = ((q < 4 ? f.x >> (8 * q) : f.y >> (8 * (q - 4))) & 0xffu) != 0u;
      const bool beats = kDesc ? (vv[q] > ve) : (vv[q] < ve);
      r += static_cast<int>(fl & (beats | ((vv[q] == ve) & (j0 + q < e))));
    }
  }
  return flag[e] ? r : 0;
}

template <bool kDesc>
__device__ __forceinline__ void rank_all(const double* v, const uint8_t* flag, int E, int* rank, int* part_cnt,
                                         int tid) {
  const int parts = rank_parts(E);
  for (int item = tid; item < E * parts; item += kSelThreads) part_cnt[item] = rank_item<kDesc>(v, flag, E, parts, item);
  __syncthreads();
  if (tid < E) {
    int r = 0;
    for (int q = 0; q < parts; ++q) r += part_cnt[q * E + tid];
    rank[tid] = r;
  }
}

// Rank counts of the n compacted values pval[i] (expert plist[i]) in (value
// desc, expert asc) order: item = (slice q, entry i) counts the entries of
// slice q that come before entry i and adds that into cnt[i] (integer LDS
// atomics, so the order of the adds does not matter).
__device__ __forceinline__ void rank_compact(const double* pval, const int* plist, int n, int* cnt, int first,
                                             int stride) {
  const int parts = max(1, (n + 15) / 16);
  const int span = (n + parts - 1) / parts;
  for (int item = first; item < n * parts; item += stride) {
    const int q = item / n, i = item % n;
    const double vi = pval[i];
    const int ei = plist[i];
    const int j_end = min(n, (q + 1) * span);
    int r = 0;
    for (int j = q * span; j < j_end; ++j) {
      const double vj = pval[j];
      r += static_cast<int>((vj > vi) | ((vj == vi) & (plist[j] < ei)));
    }
    if (r) atomicAdd(&cnt[i], r);
  }
}

// Workgroup counters without contention: each wave adds its ballot count (or
// its lane sum) with a single LDS atomic.  Integer sums, so the order of the
// atomics does not change the result.
__device__ __forceinline__ void wg_count(bool pred, int* counter, int lane) {
  const int c = popc64(__ballot(pred));
  if (lane == 0 && c) atomicAdd(counter, c);
}

__device__ __forceinline__ void wg_add(int v, int* counter, int lane) {
  const int s = wave_sum_i32(v);
  if (lane == 0 && s) atomicAdd(counter, s);
}

template <int EPL>
__device__ __forceinline__ void load_row(const float* __restrict__ zrow, int E, int lane, float (&zv)[EPL]) {
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane + kWave * i;
    zv[i] = e < E ? zrow[e] : -INFINITY;
  }
}

// ---------------------------------------------------------------------------
// natural top-k and router probabilities of NN nodes t[j] (one wave).  The
// caller loads the logit rows into zv.  emit(j, slot, e, r) stores node j's
// entry of rank `slot`.
// ---------------------------------------------------------------------------
template <int EPL, int NN, class Emit>
__device__ __forceinline__ void natural_nodes(const SelectParams& p, const int (&t)[NN], const float (&zv)[NN][EPL],
                                              int lane, NodeSlot* const (&sl)[NN], Emit&& emit) {
  const int E = p.E, k = p.k;
  uint32_t key[NN][EPL];
  double ex[NN][EPL];
  double den[NN];
#pragma unroll
  for (int j = 0; j < NN; ++j) {
#pragma unroll
    for (int i = 0; i < EPL; ++i) key[j][i] = (lane + kWave * i) < E ? logit_key(zv[j][i]) : 0u;
    // softmax over all E in fp64 (max subtracted)
    float zmax = zv[j][0];
#pragma unroll
    for (int i = 1; i < EPL; ++i) zmax = fmaxf(zmax, zv[j][i]);
    zmax = wave_max_f32(zmax);
    den[j] = 0.0;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      ex[j][i] = (lane + kWave * i) < E ? exp(static_cast<double>(zv[j][i]) - static_cast<double>(zmax)) : 0.0;
      den[j] += ex[j][i];
    }
    den[j] = wave_sum_f64(den[j]);
  }
  if (p.mode == MODE_MOESPEC) {
#pragma unroll
    for (int j = 0; j < NN; ++j)
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        const int e = lane + kWave * i;
        if (e < E) p.ws_rfull[static_cast<size_t>(t[j]) * E + e] = ex[j][i] / den[j];
      }
  }
  uint32_t thr[NN];
  kth_largest<EPL, NN>(key, k, thr);
#pragma unroll
  for (int j = 0; j < NN; ++j) {
    NodeSlot& s = *sl[j];
    const int n = topk_compact<EPL>(thr[j], key[j], k, lane, s.sk, s.se, [&](int pos, int i) { s.sx[pos] = ex[j][i]; });
    if (lane < n) emit(j, slot_of(lane, n, s.sk, s.se), s.se[lane], s.sx[lane] / den[j]);
  }
  wave_lds_sync();  // the scratch is reused by the wave's next nodes
}

template <int EPL>
__global__ __launch_bounds__(kNodeWaves * kWave) void natural_kernel(SelectParams p) {
  __shared__ NodeScratch ns;
  const int wave = wave_id(), lane = lane_id();
  const int t = blockIdx.x * kNodeWaves + wave;
  if (t >= p.T) return;
  const int tt[1] = {t};
  float zv[1][EPL];
  load_row<EPL>(p.logits + static_cast<size_t>(t) * p.E, p.E, lane, zv[0]);
  NodeSlot* const sl[1] = {&ns.s[wave]};
  natural_nodes<EPL, 1>(p, tt, zv, lane, sl, [&](int, int slot, int e, double r) {
    p.ws_kidx[static_cast<size_t>(t) * p.k + slot] = e;
    p.ws_r[static_cast<size_t>(t) * p.k + slot] = r;
  });
}

// ---------------------------------------------------------------------------
// restricted top-k over the eligible set and renormalised gates of NN nodes
// of one tree (one wave).  elig[e] != 0 marks e in S'.  Nodes with live[j]
// false are computed and not written.  Experts that receive a node are marked
// in `routed` (an LDS bitmask).
// ---------------------------------------------------------------------------
template <int EPL, int NN>
__device__ __forceinline__ void restricted_nodes(const SelectParams& p, const int (&t)[NN], const bool (&live)[NN],
                                                 const float (&zv)[NN][EPL], const uint8_t* elig, int lane,
                                                 NodeSlot* const (&sl)[NN], uint32_t* routed) {
  const int E = p.E, k = p.k;
  uint32_t key[NN][EPL];
#pragma unroll
  for (int j = 0; j < NN; ++j)
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = lane + kWave * i;
      key[j][i] = (e < E && elig[e]) ? logit_key(zv[j][i]) : 0u;
    }
  uint32_t thr[NN];
  kth_largest<EPL, NN>(key, k, thr);
#pragma unroll
  for (int j = 0; j < NN; ++j) {
    NodeSlot& s = *sl[j];
    const int n = topk_compact<EPL>(thr[j], key[j], k, lane, s.sk, s.se, [&](int pos, int i) { s.sz[pos] = zv[j][i]; });
    // gates: softmax over the selected logits, fp64
    double zm = lane < n ? static_cast<double>(s.sz[lane]) : -INFINITY;
    zm = wave_max_f64(zm);
    const double w = lane < n ? exp(static_cast<double>(s.sz[lane]) - zm) : 0.0;
    const double ws = wave_sum_f64(w);
    if (!live[j]) continue;
    int32_t* orow = p.topk_idx + static_cast<size_t>(t[j]) * k;
    float* grow = p.topk_gate + static_cast<size_t>(t[j]) * k;
    if (lane < n) {
      const int slot = slot_of(lane, n, s.sk, s.se);
      const int e = s.se[lane];
      orow[slot] = e;
      grow[slot] = static_cast<float>(w / ws);
      atomicOr(&routed[e >> 5], 1u << (e & 31));
    } else if (lane < k) {
      orow[lane] = -1;  // fewer eligible experts than k (an invalid tree has none)
      grow[lane] = 0.0f;
    }
  }
  wave_lds_sync();  // the scratch is reused by the wave's next nodes
}

// Number of list entries j2 < n ordered before entry j of value vj: larger
// (kDesc) or smaller values first, equal values by position.  Reads eight
// broadcast values per step; entries past n (stale, never beyond the
// kMaxExperts-entry list) are masked out.
template <bool kDesc>
__device__ __forceinline__ int count_before(const double* v, int n, double vj, int j) {
  int r = 0;
  for (int j0 = 0; j0 < n; j0 += 8) {
    const double2 a = *reinterpret_cast<const double2*>(v + j0);
    const double2 b = *reinterpret_cast<const double2*>(v + j0 + 2);
    const double2 c = *reinterpret_cast<const double2*>(v + j0 + 4);
    const double2 d = *reinterpret_cast<const double2*>(v + j0 + 6);
    const double vv[8] = {a.x, a.y, b.x, b.y, c.x, c.y, d.x, d.y};
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const bool beats = kDesc ? (vv[q] > vj) : (vv[q] < vj);
      r += static_cast<int>((j0 + q < n) & (beats | ((vv[q] == vj) & (j0 + q < j))));
    }
  }
  return r;
}

// ---------------------------------------------------------------------------
// Eq. 6, Sec. 3.3 and Eq. 7 for the self-sizing and fixed-budget modes, run
// by one wave (lane l holds experts l, l + 64, ...) in two parts around one
// workgroup barrier: eligible_take_wave finds n_er and the number of R
// members S takes while the other waves rank the positive members of R
// (rank_compact over the list P3 compacts); eligible_set_wave then builds S
// from those ranks,
// |S|, a(S) and the Eq. 7 pruning.  Sums take the same per-lane order and
// wave reduction as the workgroup path, integer counts are order-free, so the
// results are the same.
// ---------------------------------------------------------------------------
template <int EPL>
__device__ void eligible_take_wave(SelShared& sh, int mode, int E, int k, int bud, int lane) {
  const int kmin = min(k, E);
  const int n_anchor = sh.n_anchor, n_R = sh.n_R, n_pos = sh.n_pos;
  int ner, take;
  if (mode == MODE_SELF) {
    double u[EPL];
    bool ok[EPL], inR[EPL];
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const int e = lane + kWave * i;
      ok[i] = e < E;
      u[i] = ok[i] ? sh.u[e] : 0.0;
      inR[i] = ok[i] && sh.inR[e];
    }
    // Z = sum over R of u^+ ; H = -sum q log q ; n_er = ceil(exp(H) - 1e-9)   (Eq. 6)
    double zp = 0.0;
#pragma unroll
    for (int i = 0; i < EPL; ++i)
      if (ok[i]) zp += (inR[i] && u[i] > 0.0) ? u[i] : 0.0;
    const double Z = wave_sum_f64(zp);
    double hp = 0.0;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      if (!ok[i]) continue;
      const double uu = (inR[i] && u[i] > 0.0) ? u[i] : 0.0;
      double term = 0.0;
      if (uu > 0.0 && Z > 0.0) {
        const double q = uu / Z;
        term = q * log(q);
      }
      hp += term;
    }
    const double hs = wave_sum_f64(hp);
    ner = 0;
    if (Z > 0.0) {
      const double x = exp(-hs);
      ner = static_cast<int>(ceil(x - 1e-9));
      if (ner < 1) ner = 1;
      if (ner > n_pos) ner = n_pos;
    }
    take = ner;
    if (n_anchor + take < kmin) take = kmin - n_anchor;  // |S| >= k
    if (take > n_R) take = n_R;
  } else {
    take = bud - n_anchor;
    if (take < 0) take = 0;
    if (take > n_R) take = n_R;
    ner = take;
  }
  if (lane == 0) {
    sh.n_er = ner;
    sh.n_take = take;
  }
}

// Writes inS, inSp, rankv (pruning order, -1 outside C), pv and the scalars
// |S|, a(S), |C|, m*.  On entry plist / pval hold the positive members of R
// and pv their ranks (rank_compact).
template <int EPL>
__device__ void eligible_set_wave(SelShared& sh, int E, int k, int removal_cap, bool prune, int lane) {
  const int take = sh.n_take;
  double u[EPL];
  bool ok[EPL], inR[EPL], inS[EPL];
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane + kWave * i;
    ok[i] = e < E;
    u[i] = ok[i] ? sh.u[e] : 0.0;
    inR[i] = ok[i] && sh.inR[e];
    if (ok[i]) {
      sh.inS[e] = sh.anchor[e];
      sh.rankv[e] = -1;
    }
  }
  // S = A u first `take` of R in (u desc, index asc) order: members with u > 0
  // by their rank among themselves, then u = 0 members in index order if needed
  const int np = sh.n_pos;
  wave_lds_sync();  // inS reset above before the members are set
  for (int i = lane; i < np; i += kWave)
    if (sh.pv[i] < take) sh.inS[sh.plist[i]] = 1;
  if (take > np) {
    int base = 0;
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const bool f = inR[i] && !(u[i] > 0.0);
      const uint64_t m = __ballot(f);
      if (f && np + base + popc64(m & lanes_below(lane)) < take) sh.inS[lane + kWave * i] = 1;
      base += popc64(m);
    }
  }
  wave_lds_sync();
  // |S|, a(S) = votes of the experts outside S
  int ns = 0, as = 0;
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane + kWave * i;
    inS[i] = ok[i] && sh.inS[e] != 0;
    ns += inS[i] ? 1 : 0;
    as += (ok[i] && !inS[i]) ? sh.votes[e] : 0;
  }
  const int nS = wave_sum_i32(ns), aS = wave_sum_i32(as);
  int m_star = 0, nC = 0;
  if (prune) {
    // C = nonresident members of S ordered by (u asc, index asc)   (Sec. 3.4)
#pragma unroll
    for (int i = 0; i < EPL; ++i) {
      const bool f = inS[i] && !sh.resident[lane + kWave * i];
      const uint64_t m = __ballot(f);
      if (f) {
        const int pos = nC + popc64(m & lanes_below(lane));
        sh.plist[pos] = lane + kWave * i;
        sh.pval[pos] = u[i];
      }
      nC += popc64(m);
    }
    wave_lds_sync();
    for (int j0 = 0; j0 < nC; j0 += kWave) {
      const int j = j0 + lane;
      const double vj = j < nC ? sh.pval[j] : 0.0;
      const int r = count_before<false>(sh.pval, nC, vj, j);
      if (j < nC) {
        const int e = sh.plist[j];
        sh.rankv[e] = r;
        sh.pv[r] = sh.votes[e];
      }
    }
    wave_lds_sync();
    // m* = longest prefix with sum v <= a(S), |S| - m >= k, m <= removal cap   (Eq. 7);
    // votes are >= 0, so the prefix sums only grow and the admissible m form a prefix
    int limit = nC;
    if (nS - k < limit) limit = nS - k;
    if (removal_cap < limit) limit = removal_cap;
    if (limit < 0) limit = 0;
    int base = 0;
    for (int r0 = 0; r0 < limit; r0 += kWave) {
      const int r = r0 + lane;
      const int v = r < limit ? sh.pv[r] : 0;
      const int cum = base + wave_incl_scan_i32(v);
      const int cnt = popc64(__ballot(r < limit && cum <= aS));
      m_star += cnt;
      if (cnt < min(kWave, limit - r0)) break;
      base = lane_value(cum, kWave - 1);
    }
  }
#pragma unroll
  for (int i = 0; i < EPL; ++i) {
    const int e = lane + kWave * i;
    if (ok[i]) {
      const int rk = sh.rankv[e];
      sh.inSp[e] = inS[i] && !(rk >= 0 && rk < m_star);
    }
  }
  if (lane == 0) {
    sh.n_S = nS;
    sh.budget_a = aS;
    sh.n_C = nC;
    sh.m_star = m_star;
  }
}

// ---------------------------------------------------------------------------
// tree stage of one tree, in phases
// ---------------------------------------------------------------------------
struct TreeCtx {
  int b, t_begin, Tb, tid, wave, lane;
  int my_d;     // depth of node tid (tid < Tb)
  float my_p;   // its commitment probability
};

// P1: LDS state, the node inputs (thread tid reads node tid), tree checks and
// depth counts N_d.  The caller synchronizes before tree_code.
__device__ __forceinline__ void tree_p1(SelShared& sh, const SelectParams& p, TreeCtx& c) {
  const int tid = c.tid, Tb = c.Tb, t_begin = c.t_begin, E = p.E;
  const bool has_mask = p.resident != nullptr;
  if (tid == 0) {
    sh.code = Tb > 0 ? 0x7fffffff : CODE_EMPTY;
    sh.n_anchor = sh.n_unat = sh.n_R = sh.n_pos = sh.n_S = sh.n_C = sh.n_Sp = sh.n_routed = 0;
    sh.budget_a = sh.m_star = sh.n_er = sh.n_take = 0;
  }
  for (int i = tid; i < kMaxTreeNodes; i += kSelThreads) sh.Nd[i] = 0;
  for (int e = tid; e < kMaxExperts; e += kSelThreads) {
    sh.votes[e] = 0;
    sh.rankv[e] = 0;
    sh.anchor[e] = sh.inR[e] = sh.inS[e] = sh.inC[e] = sh.inSp[e] = sh.routed[e] = 0;
    sh.u[e] = 0.0;
    sh.score[e] = 0.0;
    sh.resident[e] = (e < E) ? (has_mask ? (p.resident[e] != 0) : 1) : 0;
  }
  c.my_d = -1;
  c.my_p = 0.0f;
  if (tid < Tb) {
    const int t = t_begin + tid;
    c.my_d = p.depth[t];
    c.my_p = p.prob[t];
    const int my_d = c.my_d;
    const float my_p = c.my_p;
    const int par = p.parent != nullptr ? p.parent[t] : 0;
    const int par_d = (p.parent != nullptr && tid > 0 && par >= t_begin && par < t) ? p.depth[par] : 0;
    int code = 0;
    if (tid == 0) {
      if (my_d != 0 || (p.parent != nullptr && par != -1)) code = CODE_ROOT;
    } else if (p.parent != nullptr) {
      if (par < t_begin || par >= t) code = CODE_PARENT;
      else if (my_d != par_d + 1) code = CODE_DEPTH;
    } else if (my_d < 1 || my_d >= Tb) {
      code = CODE_DEPTH;
    }
    if (!(my_p >= 0.0f) || !isfinite(my_p)) code = code ? code : CODE_PROB;
    if (code) atomicMin(&sh.code, code);
    if (my_d >= 0 && my_d < Tb) atomicAdd(&sh.Nd[my_d], 1);
  }
}

__device__ __forceinline__ int tree_code(const SelShared& sh) { return sh.code == 0x7fffffff ? 0 : sh.code; }

// invalid tree: an empty eligible set, so its nodes get no routing
__device__ __forceinline__ void tree_invalid(const SelectParams& p, const TreeCtx& c, int code) {
  for (int e = c.tid; e < p.E; e += kSelThreads) p.eligible[static_cast<size_t>(c.b) * p.E + e] = 0;
  if (p.stats != nullptr && c.tid < kNumStats) {
    int v = 0;
    if (c.tid == 0) v = c.Tb;
    if (c.tid == 8) v = code;
    p.stats[c.b * kNumStats + c.tid] = v;
  }
}

// alpha_t = p_t^beta / sqrt(N_{d_t})   (Eq. 3); the caller synchronizes
__device__ __forceinline__ void tree_alpha(SelShared& sh, const SelectParams& p, const TreeCtx& c) {
  if (c.tid < c.Tb) {
    const double pd = static_cast<double>(c.my_p);
    const double pb = p.beta == 0.5 ? sqrt(pd) : (p.beta == 1.0 ? pd : pow(pd, p.beta));
    sh.alpha[c.tid] = pb / sqrt(static_cast<double>(sh.Nd[c.my_d]));
  }
}

// P3: votes, anchor and the utility in node order.  kidx / rr hold the
// tree's natural entries, node tl's slot j at tl * k + j.  With kPre the
// first chunk's entry tid was loaded beforehand into (pf_e, pf_r).
template <bool kPre>
__device__ __forceinline__ void tree_p3(SelShared& sh, const SelectParams& p, const TreeCtx& c,
                                        const int32_t* kidx, const double* rr, int pf_e, double pf_r) {
  const int tid = c.tid, lane = c.lane, Tb = c.Tb, E = p.E, k = p.k;
  const int chunk = kDenseDoubles / E;  // >= 8 for E <= 512
  double u_acc = 0.0;
  for (int c0 = 0; c0 < Tb; c0 += chunk) {
    const int cn = min(chunk, Tb - c0);
    for (int i = tid; i < cn * E; i += kSelThreads) sh.dense[i] = 0.0;
    __syncthreads();
    for (int i = tid; i < cn * k; i += kSelThreads) {
      const int tl = c0 + i / k;
      const int gi = c0 * k + i;
      const bool pf = kPre && c0 == 0 && i == tid;  // loaded at the start
      const int e = pf ? pf_e : kidx[gi];
      sh.dense[(tl - c0) * E + e] = sh.alpha[tl] * (pf ? pf_r : rr[gi]);
      atomicAdd(&sh.votes[e], 1);
      if (tl == 0) sh.anchor[e] = 1;  // the root is the tree's only depth-0 node
    }
    __syncthreads();
    if (tid < E) {
#pragma unroll 8
      for (int j = 0; j < cn; ++j) u_acc += sh.dense[j * E + tid];
    }
    __syncthreads();
  }
  const bool in_e = tid < E;
  const bool anc = in_e && sh.anchor[tid];
  if (in_e) {
    sh.u[tid] = u_acc;
    sh.inR[tid] = !anc;
  }
  wg_count(anc, &sh.n_anchor, lane);
  wg_count(in_e && sh.votes[tid] > 0, &sh.n_unat, lane);
  wg_count(in_e && !anc, &sh.n_R, lane);
  // the positive members of R, compacted (in no particular order) into
  // plist / pval for the ranking of P4, with their rank counters pv zeroed;
  // n_pos is their number
  const bool pos = in_e && !anc && u_acc > 0.0;
  const uint64_t pm = __ballot(pos);
  int pbase = 0;
  if (lane == 0 && pm != 0ull) pbase = atomicAdd(&sh.n_pos, popc64(pm));
  pbase = __builtin_amdgcn_readfirstlane(pbase);
  if (pos) {
    const int i = pbase + popc64(pm & lanes_below(lane));
    sh.plist[i] = tid;
    sh.pval[i] = u_acc;
    sh.pv[i] = 0;
  }
}

// P4 and the tree's outputs: S' into sh.inSp and eligible[b], statistics
// (routed experts left 0).  Ends synchronized.
template <int EPL>
__device__ __forceinline__ void tree_p4(SelShared& sh, const SelectParams& p, const TreeCtx& c) {
  const int tid = c.tid, wave = c.wave, lane = c.lane, Tb = c.Tb, t_begin = c.t_begin, E = p.E, k = p.k;
  const int mode = p.mode;
  const int kmin = min(k, E);
  const int bud = p.budget < kmin ? kmin : (p.budget > E ? E : p.budget);

  if (mode == MODE_SELF || mode == MODE_FIXED) {
    // Eq. 6 in wave 0 while the other waves rank the positive members of R;
    // then S, |S|, a(S) and the Eq. 7 pruning in wave 0
    if (wave == 0)
      eligible_take_wave<EPL>(sh, mode, E, k, bud, lane);
    else
      rank_compact(sh.pval, sh.plist, sh.n_pos, sh.pv, tid - kWave, kSelThreads - kWave);
    __syncthreads();
    if (wave == 0) eligible_set_wave<EPL>(sh, E, k, p.removal_cap, p.resident != nullptr, lane);
    __syncthreads();
  } else {
    if (mode == MODE_MOESPEC || mode == MODE_COUNT) {
      // MoE-Spec: router mass summed over the block; Count-B: natural votes
      if (tid < E) {
        double score = 0.0;
        if (mode == MODE_MOESPEC) {
#pragma unroll 8
          for (int tl = 0; tl < Tb; ++tl) score += p.ws_rfull[static_cast<size_t>(t_begin + tl) * E + tid];
        } else {
          score = static_cast<double>(sh.votes[tid]);
        }
        sh.score[tid] = score;
        sh.inC[tid] = 1;  // every expert competes
      }
      __syncthreads();
      rank_all<true>(sh.score, sh.inC, E, sh.rankv, sh.rpart, tid);
      __syncthreads();
      if (tid < E) sh.inS[tid] = sh.rankv[tid] < bud;
    } else {  // natural routing: S = [E]
      if (tid < E) sh.inS[tid] = 1;
    }
    __syncthreads();
    // |S|, a(S)
    {
      const bool in_e = tid < E;
      const bool inS = in_e && sh.inS[tid];
      wg_count(inS, &sh.n_S, lane);
      wg_add((in_e && !inS) ? sh.votes[tid] : 0, &sh.budget_a, lane);
      wg_count(mode != MODE_ALL && inS && !sh.anchor[tid], &sh.n_er, lane);
      if (in_e) sh.inSp[tid] = inS;  // no pruning outside the self-sizing / fixed-budget modes
    }
    __syncthreads();
    if (mode == MODE_ALL && tid == 0) {
      sh.n_er = E - sh.n_anchor;
      sh.budget_a = 0;
    }
  }
  __syncthreads();

  if (tid < E) p.eligible[static_cast<size_t>(c.b) * E + tid] = sh.inSp[tid];
  wg_count(tid < E && sh.inSp[tid], &sh.n_Sp, lane);
  __syncthreads();
  if (p.stats != nullptr && tid == 0) {
    int32_t* st = p.stats + c.b * kNumStats;
    st[0] = Tb;
    st[1] = sh.n_anchor;
    st[2] = sh.n_er;
    st[3] = sh.n_S;
    st[4] = sh.n_Sp;
    st[5] = sh.n_unat;
    st[6] = sh.budget_a;
    st[7] = sh.m_star;
    st[8] = 0;
    st[9] = 0;  // routed experts, counted by the restricted stage
  }
}

__device__ __forceinline__ TreeCtx tree_ctx(const TreeOffsets& offs, int b) {
  TreeCtx c;
  c.b = b;
  c.t_begin = offs.o[b];
  c.Tb = offs.o[b + 1] - c.t_begin;
  c.tid = threadIdx.x;
  c.wave = wave_id();
  c.lane = lane_id();
  c.my_d = -1;
  c.my_p = 0.0f;
  return c;
}

// ---------------------------------------------------------------------------
// eligible set of one tree
// ---------------------------------------------------------------------------
template <int EPL>
__global__ __launch_bounds__(kSelThreads) void tree_kernel(SelectParams p, TreeOffsets offs) {
  __shared__ SelShared sh;
  TreeCtx c = tree_ctx(offs, blockIdx.x);
  const int tid = c.tid, k = p.k;
  if (tid < kRoutedWords) p.ws_routed[c.b * kRoutedWords + tid] = 0u;
  // the first utility chunk's natural top-k entries, loaded now so their
  // latency overlaps the node loads of P1
  const int32_t* kidx = p.ws_kidx + static_cast<size_t>(c.t_begin) * k;
  const double* rr = p.ws_r + static_cast<size_t>(c.t_begin) * k;
  int pf_e = 0;
  double pf_r = 0.0;
  if (tid < min(kDenseDoubles / p.E, c.Tb) * k) {
    pf_e = kidx[tid];
    pf_r = rr[tid];
  }
  tree_p1(sh, p, c);
  __syncthreads();
  const int code = tree_code(sh);
  if (code != 0) {
    tree_invalid(p, c, code);
    return;
  }
  tree_alpha(sh, p, c);
  __syncthreads();
  tree_p3<true>(sh, p, c, kidx, rr, pf_e, pf_r);
  __syncthreads();
  tree_p4<EPL>(sh, p, c);
}

// ---------------------------------------------------------------------------
// restricted top-k, one wave per node
// ---------------------------------------------------------------------------
// Routed experts are counted per tree into stats[b][9]: each wave marks its
// node's experts in an LDS bitmask; the masks of the workgroup's nodes are
// merged per tree and added to the tree's workspace bitmask with one atomic
// per nonzero word, and the newly set bits with one atomic per tree (per-slot
// global atomics on a handful of words serialize).
template <int EPL>
__global__ __launch_bounds__(kNodeWaves * kWave) void restricted_kernel(SelectParams p, TreeOffsets offs) {
  __shared__ NodeScratch ns;
  __shared__ uint32_t routed[kNodeWaves][kRoutedWords];
  __shared__ int tree_of[kNodeWaves];
  const int wave = wave_id(), lane = lane_id();
  const int t = blockIdx.x * kNodeWaves + wave;
  if (lane < kRoutedWords) routed[wave][lane] = 0u;
  int b = -1;
  if (t < p.T) {
    // tree of node t: the b with o[b] <= t < o[b+1] (empty trees are skipped)
    int lo = 0, hi = p.B - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (offs.o[mid] <= t) lo = mid;
      else hi = mid - 1;
    }
    b = lo;
    wave_lds_sync();
    const int tt[1] = {t};
    const bool live[1] = {true};
    float zv[1][EPL];
    load_row<EPL>(p.logits + static_cast<size_t>(t) * p.E, p.E, lane, zv[0]);
    NodeSlot* const sl[1] = {&ns.s[wave]};
    restricted_nodes<EPL, 1>(p, tt, live, zv, p.eligible + static_cast<size_t>(b) * p.E, lane, sl, routed[wave]);
  }
  if (lane == 0) tree_of[wave] = b;
  if (p.stats == nullptr) return;
  __syncthreads();
  if (wave == 0) {
    const int words = (p.E + 31) / 32;
    for (int w0 = 0; w0 < kNodeWaves; ++w0) {
      const int tb = tree_of[w0];
      bool first = tb >= 0;
      for (int w1 = 0; w1 < w0; ++w1) first = first && tree_of[w1] != tb;
      if (!first) continue;  // this tree was merged at its first wave
      uint32_t m = 0u;
      if (lane < words)
        for (int w1 = w0; w1 < kNodeWaves; ++w1)
          if (tree_of[w1] == tb) m |= routed[w1][lane];
      int fresh = 0;
      if (m != 0u) fresh = __popc(m & ~atomicOr(&p.ws_routed[tb * kRoutedWords + lane], m));
      fresh = wave_sum_i32(fresh);
      if (lane == 0 && fresh) atomicAdd(&p.stats[tb * kNumStats + 9], fresh);
    }
  }
}

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

}  // namespace

size_t select_workspace_bytes(int T, int E, int k) {
  const size_t Tt = static_cast<size_t>(T > 0 ? T : 0);
  return align256(Tt * k * sizeof(int32_t)) + align256(Tt * k * sizeof(double)) +
         align256(Tt * E * sizeof(double)) + align256(sizeof(uint32_t) * kMaxTrees * kRoutedWords);
}

void select_carve(void* ws, int T, int E, int k, SelectParams& p) {
  char* c = static_cast<char*>(ws);
  const size_t Tt = static_cast<size_t>(T > 0 ? T : 0);
  p.ws_kidx = reinterpret_cast<int32_t*>(c);
  c += align256(Tt * k * sizeof(int32_t));
  p.ws_r = reinterpret_cast<double*>(c);
  c += align256(Tt * k * sizeof(double));
  p.ws_rfull = reinterpret_cast<double*>(c);
  c += align256(Tt * E * sizeof(double));
  p.ws_routed = reinterpret_cast<uint32_t*>(c);
}

template <int EPL>
hipError_t launch_select_epl(const SelectParams& p, const TreeOffsets& offs, hipStream_t stream) {
  const int node_blocks = (p.T + kNodeWaves - 1) / kNodeWaves;
  if (node_blocks > 0) natural_kernel<EPL><<<node_blocks, kNodeWaves * kWave, 0, stream>>>(p);
  tree_kernel<EPL><<<p.B, kSelThreads, 0, stream>>>(p, offs);
  if (node_blocks > 0) restricted_kernel<EPL><<<node_blocks, kNodeWaves * kWave, 0, stream>>>(p, offs);
  return hipGetLastError();
}

// prob[t] = p_hat[depth[t]] (0 outside the table)
__global__ void commit_expand_kernel(const float* __restrict__ p_hat, int D, const int32_t* __restrict__ depth, int T,
                                     float* __restrict__ prob) {
  for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < T; t += gridDim.x * blockDim.x) {
    const int d = depth[t];
    prob[t] = (d >= 0 && d < D) ? p_hat[d] : 0.0f;
  }
}

hipError_t launch_commit_expand(const float* p_hat, int D, const int32_t* depth, int T, float* prob,
                                hipStream_t stream) {
  const int block = 256;
  const int grid = min((T + block - 1) / block, 1024);
  commit_expand_kernel<<<grid, block, 0, stream>>>(p_hat, D, depth, T, prob);
  return hipGetLastError();
}

hipError_t launch_select(const SelectParams& p, const TreeOffsets& offs, hipStream_t stream) {
  const int epl = (p.E + kWave - 1) / kWave;
  if (epl <= 1) return launch_select_epl<1>(p, offs, stream);
  if (epl <= 2) return launch_select_epl<2>(p, offs, stream);
  if (epl <= 4) return launch_select_epl<4>(p, offs, stream);
  return launch_select_epl<8>(p, offs, stream);
}

}  // namespace amoe

// ---------------------------------------------------------------------------
// Allocation-free selection: the same kernels with their scratch in a static
// device array instead of a caller workspace.  Each device holds its own copy
// of the array (module load) until the process ends; its address is looked up
// once per device, with that device current, and only that address is passed
// to kernels (the array's name is a host-side stand-in in host code).
// ---------------------------------------------------------------------------
namespace {

constexpr size_t kNoallocScratchBytes = ACCEPTMOE_SELECT_NOALLOC_MAX_WORKSPACE;
static_assert(kNoallocScratchBytes % 256 == 0, "scratch size keeps 256-byte carving");

static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// device address of `scratch` on the device the stream runs on (which must be
// the current device)
int32_t scratch_address(hipStream_t stream, void** out) {
  using amoe::abi::fail;
  using amoe::abi::hip_fail;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "select_noalloc: hipGetDevice");
  if (stream != nullptr) {
    hipDevice_t sdev = 0;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return hip_fail(e, "select_noalloc: hipStreamGetDevice");
    if (static_cast<int>(sdev) != dev)
      return fail(ACCEPTMOE_ERR_INVALID_ARG, "select_noalloc: the stream belongs to device %d, device %d is current",
                  static_cast<int>(sdev), dev);
  }
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED, "select_noalloc: device index %d beyond %d", dev, kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "select_noalloc: hipGetSymbolAddress(scratch)");
    if (ptr == nullptr) return fail(ACCEPTMOE_ERR_HIP, "select_noalloc: null scratch address");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return ACCEPTMOE_OK;
}

}  // namespace

extern "C" int32_t acceptmoe_select_noalloc(const float* logits, const int32_t* parent, const int32_t* depth,
                                            const float* commit_prob, const int32_t* tree_offsets, int32_t B,
                                            int32_t T, int32_t E, int32_t k, double beta, int32_t mode,
                                            int32_t budget, int32_t removal_cap, const uint8_t* resident_mask,
                                            uint8_t* eligible, int32_t* topk_idx, float* topk_gate,
                                            int32_t* stats, void* stream) {
  using amoe::abi::fail;
  using amoe::abi::hip_fail;
  amoe::abi::clear_err();
  amoe::SelectParams p;
  amoe::TreeOffsets offs;
  bool noop = false;
  int32_t rc = amoe::select_prepare("select_noalloc", logits, parent, depth, commit_prob, tree_offsets, B, T, E, k,
                                    beta, mode, budget, removal_cap, resident_mask, eligible, topk_idx, topk_gate,
                                    stats, p, offs, noop);
  if (rc != ACCEPTMOE_OK || noop) return rc;
  const size_t need = amoe::select_workspace_bytes(T, E, k);
  if (need > kNoallocScratchBytes)
    return fail(ACCEPTMOE_ERR_UNSUPPORTED,
                "select_noalloc: T=%d E=%d k=%d needs %zu bytes of scratch, beyond the static %zu bytes "
                "(use acceptmoe_select with a workspace)", T, E, k, need, kNoallocScratchBytes);
  void* ws = nullptr;
  rc = scratch_address(static_cast<hipStream_t>(stream), &ws);
  if (rc != ACCEPTMOE_OK) return rc;
  amoe::select_carve(ws, T, E, k, p);
  hipError_t e = amoe::launch_select(p, offs, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? ACCEPTMOE_OK : hip_fail(e, "select_noalloc launch");
}

