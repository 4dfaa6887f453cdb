/*
 * acceptmoe.h -- C ABI of the MI355X (gfx950) verify-block MoE layer.
 *
 * The layer follows "AcceptMoE: Commitment-Weighted Self-Sizing Verifier
 * Expert Sets for Efficient MoE Speculative Decoding" (arXiv 2608.02989):
 * one MoE layer of one speculative-decoding verification block, with the
 * eligible expert set chosen from commitment-weighted router demand.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All tensor pointers are DEVICE pointers owned by the caller, row-major
 *    and contiguous, unless an argument says "host".  The library allocates
 *    no device memory and keeps no state between calls.
 *  - Every call is asynchronous on `stream` (a hipStream_t passed as void*,
 *    NULL = the default stream) and never synchronises the host, so a whole
 *    route -> select -> forward sequence can be captured in a HIP graph.
 *  - Return value: ACCEPTMOE_OK (0) or a negative ACCEPTMOE_ERR_* code.  All
 *    argument checks run on the host before any HIP call, so a rejected call
 *    launches nothing and touches no memory.  acceptmoe_last_error() then
 *    returns a thread-local, human-readable reason.
 *  - Contents of device arrays (tree structure, probabilities, routing
 *    indices) are checked by the kernels themselves: malformed trees are
 *    reported through `stats`, out-of-range routing indices are skipped.
 *    Logits or activations that are NaN or Inf give unspecified (but
 *    memory-safe) results.
 *  - Calls that share a workspace must be stream-ordered.
 */
#ifndef ACCEPTMOE_H
#define ACCEPTMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define ACCEPTMOE_OK 0
#define ACCEPTMOE_ERR_INVALID_ARG (-1) /* null pointer, bad size, bad enum      */
#define ACCEPTMOE_ERR_UNSUPPORTED (-2) /* shape outside the supported limits    */
#define ACCEPTMOE_ERR_WORKSPACE (-3)   /* workspace pointer/size too small      */
#define ACCEPTMOE_ERR_HIP (-4)         /* a HIP launch or runtime call failed   */

/* element types */
#define ACCEPTMOE_F32 0
#define ACCEPTMOE_BF16 1

/* eligible-set rules (acceptmoe_select `mode`) */
#define ACCEPTMOE_MODE_SELF_SIZING 0  /* AcceptMoE: anchor + effective rank (Sec. 3.3)   */
#define ACCEPTMOE_MODE_ALL_EXPERTS 1  /* S = [E]: natural routing, Standard SD (Sec. 3.1) */
#define ACCEPTMOE_MODE_FIXED_BUDGET 2 /* AcceptMoE-B: anchor + top of R by u, |S| = B (Sec. 4) */
#define ACCEPTMOE_MODE_MOESPEC 3      /* top-B by summed router mass (Sec. 4 baseline)  */
#define ACCEPTMOE_MODE_COUNT 4        /* top-B by natural top-k votes (Sec. 4 baseline) */

/* per-tree statistics row written by acceptmoe_select (int32 each) */
#define ACCEPTMOE_STAT_T 0         /* nodes in the tree                            */
#define ACCEPTMOE_STAT_ANCHOR 1    /* |A|, root natural top-k (Eq. 5)              */
#define ACCEPTMOE_STAT_NER 2       /* n_er (Eq. 6) or non-anchor members taken     */
#define ACCEPTMOE_STAT_S 3         /* |S| before pruning                           */
#define ACCEPTMOE_STAT_SPRIME 4    /* |S'| after residency pruning (Eq. 7)         */
#define ACCEPTMOE_STAT_UNAT 5      /* |U_nat|, natural union (Eq. 1)               */
#define ACCEPTMOE_STAT_BUDGET 6    /* rerouting budget a(S) (Sec. 3.4)             */
#define ACCEPTMOE_STAT_MSTAR 7     /* m*, experts removed by pruning (Eq. 7)       */
#define ACCEPTMOE_STAT_CODE 8      /* 0 = ok, else ACCEPTMOE_TREE_* below          */
#define ACCEPTMOE_STAT_ROUTED 9    /* experts that receive a token of this tree    */
#define ACCEPTMOE_NUM_STATS 10

/* tree validation codes (the smallest applicable code is reported) */
#define ACCEPTMOE_TREE_OK 0
#define ACCEPTMOE_TREE_EMPTY 1       /* tree with no node                              */
#define ACCEPTMOE_TREE_BAD_ROOT 2    /* first node is not a root (parent -1, depth 0)  */
#define ACCEPTMOE_TREE_BAD_PARENT 3  /* a later node's parent is not an earlier node
                                        of the same tree                               */
#define ACCEPTMOE_TREE_BAD_DEPTH 4   /* depth != parent depth + 1 (or out of range)    */
#define ACCEPTMOE_TREE_BAD_PROB 5    /* commitment probability < 0 or not finite       */

/* supported limits */
#define ACCEPTMOE_MAX_EXPERTS 512
#define ACCEPTMOE_MAX_TOPK 32
#define ACCEPTMOE_MAX_TREES 256
#define ACCEPTMOE_MAX_TREE_NODES 1024
/* static scratch of acceptmoe_select_noalloc per device: 8 MiB (e.g. up to
 * 7,000 nodes at E = 128, k = 8; acceptmoe_select_workspace_size gives the need) */
#define ACCEPTMOE_SELECT_NOALLOC_MAX_WORKSPACE ((size_t)8 << 20)

/*
 * acceptmoe_packed_router_bytes -- bytes of a packed router matrix:
 *   ceil(E / 16) * 16 * ceil(H / 32) * 32 * 6 (0 for unsupported E or H).
 * acceptmoe_pack_router_weights -- converts the fp32 router matrix W_r
 * [E, H] (nn.Linear orientation, row-major) into the layout acceptmoe_route
 * reads.  Each weight w becomes three bf16 values (round to nearest even)
 * hi = bf16(w), mid = bf16(w - hi), lo = bf16(w - hi - mid), whose sum is w
 * exactly for 1e-33 < |w| < 3.39e38 (the largest bf16; beyond it hi is
 * infinite).  Rows are padded with zeros to a
 * multiple of 16 and columns to a multiple of 32; then for every 16-row tile
 * et, every 32-column chunk c and every plane p (0 hi, 1 mid, 2 lo) a
 * fragment of 64 lanes x 16 B follows, lane L holding plane p of row
 * 16*et + (L % 16), columns 32*c + 8*(L / 16) .. +7 (eight bf16).  Fragment
 * (et, c, p) starts at byte ((et * ceil(H/32) + c) * 3 + p) * 1024.  A
 * one-time, load-time step.
 *
 *   src  [E, H] fp32 device;  dst device, acceptmoe_packed_router_bytes(E, H)
 *   bytes, must not overlap src.  1 <= E <= ACCEPTMOE_MAX_EXPERTS,
 *   H >= 16 and H % 16 == 0; both 16-byte aligned.
 */
size_t acceptmoe_packed_router_bytes(int32_t E, int32_t H);
int32_t acceptmoe_pack_router_weights(const float* src, int32_t E, int32_t H, void* dst, void* stream);

/*
 * acceptmoe_route -- router logits z_t = W_r h_t for every node of the block
 * (Sec. 3.1, the target-router logits z_t the selector consumes).
 *
 *   hidden         [T, H] device, element type `hidden_dtype` (F32 or BF16),
 *                  16-byte aligned
 *   router_packed  W_r [E, H] in the layout of acceptmoe_pack_router_weights
 *   logits         [T, E] device fp32, written
 *   T >= 0 (T == 0 is a no-op), 1 <= E <= ACCEPTMOE_MAX_EXPERTS,
 *   H >= 16 and H % 16 == 0.
 * Products are exact (bf16 hidden times each bf16 plane, or fp32 hidden
 * times the rebuilt fp32 weight) and accumulation is fp32, so the logits
 * carry fp32 accuracy; the result is deterministic (fixed reduction order).
 */
int32_t acceptmoe_route(const void* hidden, int32_t hidden_dtype, const void* router_packed,
                        int32_t T, int32_t H, int32_t E, float* logits, void* stream);

/*
 * acceptmoe_select_workspace_size -- bytes of device workspace acceptmoe_select
 * needs for T nodes and top-k.  No alignment beyond 256 bytes is required.
 */
size_t acceptmoe_select_workspace_size(int32_t T, int32_t E, int32_t k);

/*
 * acceptmoe_select -- eligible expert set per verification tree and the
 * restricted routing of every node (Sec. 3.1-3.4, Eq. 1-7).
 *
 * Per tree b (nodes tree_offsets[b] .. tree_offsets[b+1]-1):
 *   r_t = softmax(z_t), K_t = TopK_k(z_t) (Sec. 3.1); votes v_e, U_nat (Eq. 1);
 *   alpha_t = p_t^beta / sqrt(N_{d_t}) (Eq. 3); u_e = sum_t alpha_t r_{t,e} 1[e in K_t]
 *   (Eq. 4); A = K_root (Eq. 5); n_er = ceil(exp(H(q)) - 1e-9) over R = [E] \ A
 *   (Eq. 6); S = A u Top_{n_er}(U_R), |S| >= k (Sec. 3.3); with a residency mask
 *   the longest prefix of the nonresident members ordered by (u asc, index asc)
 *   allowed by Eq. 7 is removed, giving S'; finally every node is routed by
 *   TopK_k(z_t + M_{S'}) (Eq. 2) with gates = softmax over its k selected logits.
 * Ties in logits (fp32) and in utilities (fp64) go to the lower expert index.
 *
 *   logits        [T, E] fp32 device (e.g. from acceptmoe_route)
 *   parent        [T] int32 device, global node ids, -1 for each tree's root;
 *                 NULL = not available (only depth ranges are checked)
 *   depth         [T] int32 device, draft position d_t (tree depth, or block
 *                 offset for a chain)
 *   commit_prob   [T] fp32 device, p_{d_t} per node (expand a per-depth table
 *                 p_hat[d] on the caller side)
 *   tree_offsets  [B+1] int32 HOST array: 0 = o_0 <= o_1 <= ... <= o_B = T;
 *                 NULL means one tree holding all T nodes (B must be 1).
 *                 Read during the call only.  Each tree needs
 *                 o_{b+1} - o_b <= ACCEPTMOE_MAX_TREE_NODES.
 *   B             trees, 1 <= B <= ACCEPTMOE_MAX_TREES (T == 0 with B == 0 is a no-op)
 *   k             top-k, 1 <= k <= min(E, ACCEPTMOE_MAX_TOPK)
 *   beta          commitment sharpness (paper default 0.5), finite, >= 0
 *   mode          ACCEPTMOE_MODE_*
 *   budget        |S| for the fixed-budget modes (clamped to [k, E]); ignored otherwise
 *   removal_cap   pruning removal cap (Sec. 3.4); < 0 means E (nonbinding)
 *   resident_mask [E] uint8 device, nonzero = expert resident; NULL = no pruning
 *                 (full residency).  Shared by all trees.
 *   eligible      [B, E] uint8 device, written: 1 if e in S'_b
 *   topk_idx      [T, k] int32 device, written: restricted experts of node t in
 *                 (logit desc, index asc) order; -1 for nodes of an invalid tree
 *   topk_gate     [T, k] fp32 device, written: renormalised gates (0 for -1 slots)
 *   stats         [B, ACCEPTMOE_NUM_STATS] int32 device, written; may be NULL
 *   workspace     device scratch of acceptmoe_select_workspace_size(T, E, k) bytes
 */
int32_t acceptmoe_select(const float* logits, const int32_t* parent, const int32_t* depth,
                         const float* commit_prob, const int32_t* tree_offsets, int32_t B,
                         int32_t T, int32_t E, int32_t k, double beta, int32_t mode,
                         int32_t budget, int32_t removal_cap, const uint8_t* resident_mask,
                         uint8_t* eligible, int32_t* topk_idx, float* topk_gate, int32_t* stats,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * acceptmoe_select_noalloc -- acceptmoe_select without a workspace argument,
 * for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation).  The same
 * kernels and outputs; their scratch is a static device array of
 * ACCEPTMOE_SELECT_NOALLOC_MAX_WORKSPACE bytes that every device the library
 * runs on holds from module load until the process ends.  The call allocates
 * nothing and calls no allocating routine.
 *
 *   Arguments as acceptmoe_select.  The scratch of the current device is used;
 *   `stream` must belong to that device (else ACCEPTMOE_ERR_INVALID_ARG).
 *   Calls needing more than the maximum (acceptmoe_select_workspace_size(T, E,
 *   k) > ACCEPTMOE_SELECT_NOALLOC_MAX_WORKSPACE) return ACCEPTMOE_ERR_UNSUPPORTED
 *   before any HIP call.
 *   Every call on one device shares that device's array, which keeps the last
 *   call's contents (each call writes every scratch word it reads before
 *   reading it, so nothing needs clearing); calls that overlap on one device,
 *   e.g. on two streams, race and are not allowed.
 */
int32_t acceptmoe_select_noalloc(const float* logits, const int32_t* parent, const int32_t* depth,
                                 const float* commit_prob, const int32_t* tree_offsets, int32_t B,
                                 int32_t T, int32_t E, int32_t k, double beta, int32_t mode,
                                 int32_t budget, int32_t removal_cap, const uint8_t* resident_mask,
                                 uint8_t* eligible, int32_t* topk_idx, float* topk_gate, int32_t* stats,
                                 void* stream);

/*
 * acceptmoe_packed_weights_bytes -- bytes of a packed expert-weight stack.
 * acceptmoe_pack_expert_weights -- converts a row-major stack [E, N, K]
 * (nn.Linear [out, in] per expert) into the MFMA fragment layout the expert
 * FFN streams: for every expert, every 16-row tile and every K chunk of
 * 64 bytes per row, the 16 x (64 B) block is stored as 64 lanes x 16 B, lane
 * L holding row (L % 16), bytes 16*(L / 16) .. +15 of that chunk.  Each wave
 * load of a weight fragment is then one contiguous 1 KiB read.  The packed
 * stack has exactly the size of the source.  A one-time, load-time step.
 *
 *   src  [E, N, K] device, dtype F32 or BF16;  dst packed, device, same size,
 *   must not overlap src.  Requires N % 16 == 0 and K % (64 / sizeof(elem)) == 0.
 * The down stack [E, H, I] is packed this way (N = H, K = I); the gate and
 * up stacks go through acceptmoe_pack_gate_up_weights.
 */
size_t acceptmoe_packed_weights_bytes(int32_t dtype, int32_t E, int32_t N, int32_t K);
int32_t acceptmoe_pack_expert_weights(const void* src, int32_t dtype, int32_t E, int32_t N,
                                      int32_t K, void* dst, void* stream);

/*
 * acceptmoe_packed_gate_up_bytes -- bytes of a packed gate/up pair of stacks.
 * acceptmoe_pack_gate_up_weights -- packs the gate and up stacks [E, I, H]
 * (the W_g and W_u of Eq. 2) into one buffer laid out for the gate/up pass:
 * for every expert e, every pair p of 16-row tiles (rows 32p .. 32p+31 of I)
 * and every K chunk c (64 bytes of each row), four 1 KiB fragments follow
 * each other -- gate tile 2p, gate tile 2p+1, up tile 2p, up tile 2p+1 --
 * each in the fragment order of acceptmoe_pack_expert_weights (lane L holds
 * row L % 16, bytes 16*(L / 16) .. +15 of the chunk).  Fragment
 * ((e * ceil(I/32) + p) * (H*eb/64) + c) * 4 + f starts at byte 1024 times
 * that index.  When I/16 is odd the last pair's second tiles are zeros, so the
 * size is E * ceil(I/32) * 32 * H * eb * 2 bytes (exactly the two stacks when
 * I % 32 == 0).  A one-time, load-time step.
 *
 *   w_gate, w_up  [E, I, H] device, dtype F32 or BF16 (eb = 4 or 2 bytes)
 *   dst           device, acceptmoe_packed_gate_up_bytes(dtype, E, I, H)
 *                 bytes, must not overlap either source
 *   Requires I % 16 == 0 and H % (64 / eb) == 0; pointers 16-byte aligned.
 */
size_t acceptmoe_packed_gate_up_bytes(int32_t dtype, int32_t E, int32_t I, int32_t H);
int32_t acceptmoe_pack_gate_up_weights(const void* w_gate, const void* w_up, int32_t dtype,
                                       int32_t E, int32_t I, int32_t H, void* dst, void* stream);

/*
 * acceptmoe_moe_forward_workspace_size -- device workspace bytes for
 * acceptmoe_moe_forward.
 */
size_t acceptmoe_moe_forward_workspace_size(int32_t T, int32_t H, int32_t I, int32_t E,
                                            int32_t k, int32_t dtype);

/*
 * acceptmoe_moe_forward -- grouped SwiGLU expert FFN over the restricted
 * routing (Sec. 3.1, Eq. 2: tokens are dispatched only to experts of S'):
 *   out_t = sum_j g_{t,j} W_d,e (silu(W_g,e x_t) * W_u,e x_t),  e = topk_idx[t, j].
 * Only experts that receive at least one token are read, each exactly once.
 *
 *   hidden        [T, H] device, element type `dtype`
 *   w_gate_up     gate and up stacks packed by acceptmoe_pack_gate_up_weights, `dtype`
 *   w_down        packed [E, H, I] stack (acceptmoe_pack_expert_weights), `dtype`
 *   topk_idx      [T, k] int32 device; entries outside [0, E) are skipped, and an
 *                 expert repeated within a row is used once (at its first slot)
 *   topk_gate     [T, k] fp32 device
 *   out           [T, H] fp32 device, written (every element)
 *   workspace     acceptmoe_moe_forward_workspace_size(...) bytes, 256-byte
 *                 aligned, not shared by calls that may run concurrently
 *   Limits: H % 32 == 0 and I % 32 == 0 (bf16), H % 16 == 0 and I % 16 == 0
 *   (fp32); 1 <= E <= ACCEPTMOE_MAX_EXPERTS; 1 <= k <= ACCEPTMOE_MAX_TOPK;
 *   T == 0 is a no-op.
 * bf16: MFMA bf16 products with fp32 accumulation; the SwiGLU activation is
 * rounded to bf16 before the down projection.  fp32: fp32 MFMA throughout.
 * The result is deterministic.  For T <= 256 with T*k <= 2048 the expert
 * contributions of a token are summed in a fixed expert order inside each of
 * 8 accumulation lanes, the lanes in a fixed order, and (when I is split in
 * two) the two fp32 halves added onto zero, which commutes; larger blocks sum
 * the k contributions of a token in slot order.
 */
int32_t acceptmoe_moe_forward(const void* hidden, int32_t dtype, const void* w_gate_up,
                              const void* w_down, int32_t T, int32_t H, int32_t I, int32_t E,
                              int32_t k, const int32_t* topk_idx,
                              const float* topk_gate, float* out, void* workspace,
                              size_t workspace_bytes, void* stream);

/*
 * acceptmoe_residual_add -- out = hidden + y, rounded to `dtype` (bf16: the
 * fp32 sum rounded to nearest even; fp32: the plain sum).  Chains stacked
 * verify layers: the next layer's input is the previous one's input plus its
 * MoE output (the residual stream of the target stack; attention is not part
 * of this library).  hidden and out [T, H] of `dtype` (out may equal hidden),
 * y [T, H] fp32, all device and 16-byte aligned; H % 4 == 0.
 */
int32_t acceptmoe_residual_add(const void* hidden, int32_t dtype, const float* y, int32_t T,
                               int32_t H, void* out, void* stream);

/*
 * ---------------------------------------------------------------------------
 * Offline commitment estimator (Sec. 3.2)
 * ---------------------------------------------------------------------------
 * p_hat_d = c_d / m_d over verification traces: m_d counts the proposed nodes
 * at draft position d (tree depth, or block offset for a chain), c_d those on
 * the accepted output prefix -- a marginal commitment probability.  The table
 * is fixed offline; acceptmoe_commit_expand turns it into the per-node
 * commit_prob that acceptmoe_select takes (p_t = p_hat[d_t]).
 *
 * acceptmoe_commit_count -- accumulates one block: for every node t with
 *   0 <= depth[t] < D, m[d] += 1 and c[d] += (on_path[t] != 0).  Host arrays:
 *   depth int32 [T], on_path uint8 [T], m and c int64 [D] (caller zeroes them
 *   before the first block).
 * acceptmoe_commit_estimate -- p_hat[d] = c[d] / m[d] computed in double and
 *   rounded once to float, 0 where m[d] == 0.  Host arrays; rejects c > m or
 *   negative counts.
 * acceptmoe_commit_expand -- prob[t] = p_hat[depth[t]], 0 for depths outside
 *   [0, D).  Device arrays p_hat float [D], depth int32 [T], prob float [T];
 *   asynchronous on `stream`.
 */
int32_t acceptmoe_commit_count(const int32_t* depth, const uint8_t* on_path, int32_t T, int32_t D,
                               int64_t* m, int64_t* c);
int32_t acceptmoe_commit_estimate(const int64_t* m, const int64_t* c, int32_t D, float* p_hat);
int32_t acceptmoe_commit_expand(const float* p_hat, int32_t D, const int32_t* depth, int32_t T,
                                float* prob, void* stream);

/*
 * ---------------------------------------------------------------------------
 * Physical expert offload (Sec. 3.4, offload paragraph; Sec. 4, offload setup)
 * ---------------------------------------------------------------------------
 * Each MoE layer keeps an X-slot expert pool in device memory and the packed
 * weights of all E experts in pinned host memory.  The pool limits residency,
 * not eligibility: selection sees the resident set as `resident_mask`, and an
 * expert that receives a token while not resident is copied into a slot
 * before the forward runs.  A block whose routed union exceeds X is served in
 * waves of tokens whose unions fit.  The pool state is host memory owned by
 * the caller; one state per layer; calls on one state must not overlap.
 *
 * Policy (the paper leaves these open; each is stated here):
 *   - a slot holds one expert's gate, up and down weights of the layer;
 *   - waves: tokens in node order join the current wave unless its routed
 *     union would exceed X, else they open the next wave (needs X >= k);
 *   - recency is kept per wave: each expert a wave uses is stamped with the
 *     wave's time; a load evicts the oldest slot whose expert the wave does
 *     not use (empty slots first, lower slot index on equal stamps);
 *   - a wave's experts are visited in ascending index; one access per (wave,
 *     expert), a hit when the expert is resident before the wave's loads.
 *
 * stats: int64[ACCEPTMOE_POOL_NUM_STATS], accumulated (never reset) by
 * acceptmoe_pool_serve_wave.
 */
#define ACCEPTMOE_POOL_WAVES 0     /* waves served                                 */
#define ACCEPTMOE_POOL_ACCESSES 1  /* (wave, routed expert) accesses               */
#define ACCEPTMOE_POOL_HITS 2      /* accesses that found the expert resident      */
#define ACCEPTMOE_POOL_MISSES 3    /* accesses that loaded the expert              */
#define ACCEPTMOE_POOL_H2D_BYTES 4 /* bytes copied host -> device by those loads   */
#define ACCEPTMOE_POOL_NUM_STATS 5

/*
 * acceptmoe_pool_state_bytes -- host bytes of the state of an X-slot pool over
 * E experts (0 for X < 1 or E outside [1, ACCEPTMOE_MAX_EXPERTS]).
 * acceptmoe_pool_init -- initialises `state` (8-byte aligned host memory of at
 * least that size) to an empty pool.
 */
size_t acceptmoe_pool_state_bytes(int32_t X, int32_t E);
int32_t acceptmoe_pool_init(void* state, size_t state_bytes, int32_t X, int32_t E);

/*
 * acceptmoe_pool_resident_mask -- mask[e] = 1 if expert e is in the pool, else
 * 0 (host array of E bytes): the residency mask for the next block's
 * selection (Eq. 7).
 */
int32_t acceptmoe_pool_resident_mask(const void* state, uint8_t* mask);

/*
 * acceptmoe_pool_plan_waves -- partitions the T tokens of a block into waves
 * (policy above).  topk_idx: host [T, k] routing rows (entries outside
 * [0, E) and repeats within a row are ignored); wave_of: host [T] output;
 * n_waves: host output (0 when T == 0).  ACCEPTMOE_ERR_UNSUPPORTED when a
 * single token routes to more than X experts.
 */
int32_t acceptmoe_pool_plan_waves(const int32_t* topk_idx, int32_t T, int32_t k, int32_t E,
                                  int32_t X, int32_t* wave_of, int32_t* n_waves);

/*
 * acceptmoe_pool_serve_wave -- makes every expert routed by the tokens of wave
 * `wave` resident (hits refresh recency; misses evict and load), then writes
 * slot_idx (host [T, k]): the slot of each entry's expert for the wave's
 * tokens, -1 for other tokens and for ignored entries, so that
 * acceptmoe_moe_forward over the pool (E = X experts, gates unchanged) runs
 * that wave.
 *   host_gate_up, host_down  pinned host stacks of all E experts in the
 *                            acceptmoe_pack_gate_up_weights /
 *                            acceptmoe_pack_expert_weights layouts
 *   pool_gate_up, pool_down  device pools of X slots in the same layouts
 *   gate_up_bytes, down_bytes bytes of one expert in each stack
 * Loads are hipMemcpyAsync on `stream` (stream-ordered before any later
 * launch on it).  With all four weight pointers NULL only the bookkeeping is
 * done (planning and traffic accounting without copies).
 */
int32_t acceptmoe_pool_serve_wave(void* state, const int32_t* topk_idx, const int32_t* wave_of,
                                  int32_t wave, int32_t T, int32_t k, const void* host_gate_up,
                                  const void* host_down, void* pool_gate_up, void* pool_down,
                                  size_t gate_up_bytes, size_t down_bytes, int32_t* slot_idx,
                                  int64_t* stats, void* stream);

/*
 * acceptmoe_copy_rows -- dst[t, :] = src[t, :] (fp32 [T, H] device arrays)
 * for every t with row_tag[t] == tag (device int32 [T]); other rows of dst
 * are left as they are.  Joins the outputs of a block served in waves.
 * Requires H % 4 == 0, T <= 65535, 16-byte aligned src and dst.
 */
int32_t acceptmoe_copy_rows(const float* src, float* dst, const int32_t* row_tag, int32_t tag,
                            int32_t T, int32_t H, void* stream);

/*
 * acceptmoe_stream_read -- a measurement, not part of the method: reads the
 * `bytes` bytes at src (device, 16-byte aligned, bytes % 16 == 0) with
 * 16-byte non-temporal loads, `grid` workgroups of 256 threads each taking
 * one contiguous share, and writes one XOR checksum word per workgroup to
 * sink[0 .. grid) (device uint32).  Its time gives the HBM read rate a plain
 * stream reaches on the device, the attainable counterpart of the expert-
 * weight stream of acceptmoe_moe_forward.  1 <= grid <= 65535; bytes == 0 is
 * a no-op.
 */
int32_t acceptmoe_stream_read(const void* src, size_t bytes, uint32_t* sink, int32_t grid, void* stream);

/* Thread-local description of the last error (empty string if none). */
const char* acceptmoe_last_error(void);

/* Library ABI version (major * 100 + minor). */
int32_t acceptmoe_version(void);

#ifdef __cplusplus
}
#endif

#endif /* ACCEPTMOE_H */
