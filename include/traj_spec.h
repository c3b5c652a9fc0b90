/*
 * traj_spec.h -- C ABI of libtrajspec, the MI355X (gfx950) trajectory-verification step
 * for trajectory-level speculative decoding of diffusion language models.
 *
 * One verification step of the method (Sec. 3.1 overview, stage 3) runs calls 1-3 back
 * to back on one HIP stream; call 4 (stage 2) builds the next step's drafts from its result:
 *   1. traj_verify_attn      -- attention of every draft block under the trajectory mask
 *                               (Sec. 3.3, "Attention masking for trajectory isolation").
 *   2. traj_confidence_topk  -- per-position confidence c(x) = max softmax and top-k
 *                               candidates over the vocabulary (Sec. 3.2, Eq. 2 and
 *                               "Candidate collection").
 *   3. traj_accept           -- threshold-decoding consistency of every draft with its
 *                               parent state and the greedy / longest-path walk
 *                               (Sec. 3.3, "Verification procedure"; Sec. 2.1 threshold
 *                               decoding; Alg. 1 phase 1 for the high-confidence set).
 *   4. traj_build_tree       -- the next step's draft tree from the accepted state
 *                               (Alg. 1: stratification, top-k first level, top-1 deeper,
 *                               pruning by path confidence).
 *   5. traj_interblock_trigger, traj_joint_peers and traj_verify_attn_peers -- inter-block
 *                               speculation (Sec. 3.4): the trigger, the visibility masks of
 *                               the joint trees of two blocks, and attention over them.
 *   6. traj_verify_layer     -- a whole decoder layer of the verification forward pass around
 *                               call 1 (norms, projections, RoPE, MLP; synthetic weights),
 *                               traj_refresh_layer, the same layer over whole sequences that
 *                               refreshes the dual cache at a block boundary, and traj_linear,
 *                               the projection GEMM on its own.
 *
 * Conventions shared by every entry point
 *   - Array arguments are DEVICE pointers owned by the caller, on the device that is
 *     current when the call is made.  The library never frees or retains them and
 *     allocates no device memory.
 *   - Calls validate their host-visible arguments, enqueue kernels on `stream` (a
 *     hipStream_t passed as void*; NULL = the legacy default stream) and return without
 *     synchronising.  Results are ready when the stream has reached that point.
 *   - Apart from traj_get_device_status, a call enqueues kernel launches only (no memory
 *     set, copy, allocation or synchronisation), so a sequence of calls on a stream being
 *     captured into a HIP graph can be replayed; every reduction runs in a fixed order, so
 *     a replay gives the same bits as the eager calls on the same inputs.
 *   - Errors are returned as traj_status, never thrown.  When a call returns anything but
 *     TRAJ_OK nothing was enqueued (except TRAJ_E_HIP, which reports a failed launch).
 *   - Conditions that only the device can see (a parent array that is not topological)
 *     never cause out-of-bounds accesses: the kernels treat such a parent as -1 and set a
 *     bit in a per-device status word that traj_get_device_status() reads.
 *   - bf16 means IEEE-754 binary32 truncated to its upper 16 bits (bfloat16), passed as
 *     raw 16-bit storage.  Outputs are rounded to nearest even.
 */
#ifndef TRAJ_SPEC_H
#define TRAJ_SPEC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TRAJ_OK = 0,
    TRAJ_E_NULL = 1,        /* a required pointer is NULL                              */
    TRAJ_E_SHAPE = 2,       /* a size is out of range or inconsistent                 */
    TRAJ_E_DTYPE = 3,       /* unknown element type                                   */
    TRAJ_E_UNSUPPORTED = 4, /* valid but not implemented here (e.g. head_dim 96)      */
    TRAJ_E_WORKSPACE = 5,   /* workspace too small or misaligned                      */
    TRAJ_E_HIP = 6,         /* the HIP runtime reported an error                      */
    TRAJ_E_ARG = 7          /* an enumerated argument has an unknown value            */
} traj_status;

typedef enum { TRAJ_BF16 = 0, TRAJ_F32 = 1 } traj_dtype;

/* Device status bits (traj_get_device_status). */
#define TRAJ_DEV_BAD_PARENT 0x1 /* some parent[n] was outside [-1, n): treated as -1      */
#define TRAJ_DEV_BAD_LEAF 0x2   /* traj_build_tree: a leaf outside [-1, n_prev): taken as -1 */
#define TRAJ_DEV_BAD_BLOCK 0x4  /* some block_start[b] was outside [0, S]: clamped              */
#define TRAJ_DEV_BAD_ROOT 0x8   /* traj_joint_peers: a root index outside its tree: taken as 0   */

/* ------------------------------------------------------------------------------------
 * 1. Trajectory-masked verification attention  (Sec. 3.3; drafts packed as in Sec. 3.2
 *    "Complexity analysis": one concatenated forward over all draft blocks)
 *
 * For every sequence b, draft n, block position p and query head h:
 *     out[b,n,p,h,:] = softmax_j( scale * q[b,n,p,h,:] . key_j ) * value_j
 * over the keys j VISIBLE to draft n:
 *     - all S dual-cache tokens k_cache[b,s,g,:] (prefix and suffix; frozen for the block),
 *     - all L tokens of draft n itself (bidirectional),
 *     - all L tokens of every ancestor of draft n (draft_parent chain up to -1),
 * and no token of any other draft.  g = h / (Hq / Hkv) (query heads of one K/V head are
 * contiguous).  With every parent -1 this is exactly the paper's isolation mask.
 * The softmax is taken in fp32 with fp32 accumulation; out is rounded to bf16.
 *
 * Layouts (row-major, contiguous, bf16):
 *     q, out            [B, N, L, Hq, D]
 *     k_cache, v_cache  [B, S, Hkv, D]
 *     k_draft, v_draft  [B, N, L, Hkv, D]
 *     draft_parent      [B, N] int32; -1 = child of the committed state, else parent[n] < n
 * Limits: D in {64, 128}; Hq % Hkv == 0; 1 <= N <= 64; 1 <= L; S >= 0; B >= 1;
 *         one sequence's cache slice S*Hkv*D*2 bytes below 2 GiB (else TRAJ_E_UNSUPPORTED);
 *         all pointers 16-byte aligned.  RoPE, if any, is already applied by the caller.
 * scale <= 0 selects 1/sqrt(D).
 * workspace: reserved; the attention kernels use no scratch memory and
 * traj_verify_attn_workspace_size() returns 0.  The pointer and size are ignored (NULL / 0
 * are the expected values).
 * out must not alias any input.
 * ------------------------------------------------------------------------------------ */
typedef struct {
    int32_t B, N, L, Hq, Hkv, D, S;
    float scale;
} traj_attn_shape;

size_t traj_verify_attn_workspace_size(const traj_attn_shape* shape);

traj_status traj_verify_attn(const void* q, const void* k_cache, const void* v_cache,
                             const void* k_draft, const void* v_draft,
                             const int32_t* draft_parent, void* out,
                             const traj_attn_shape* shape,
                             void* workspace, size_t workspace_bytes, void* stream);

/* traj_verify_attn with per-draft peer visibility  (Sec. 3.4 "Joint tree construction",
 * App. D: the trees of two consecutive blocks verified in one pass, each draft additionally
 * seeing the root draft of the other block's tree; traj_joint_peers builds those masks).
 * draft_peers [B, N] uint64 (device, may be NULL = traj_verify_attn): bit j of
 * draft_peers[b,n] makes all L tokens of draft j visible to draft n in addition to the cache,
 * itself and its ancestors; one direction per bit (mutual visibility sets both); bits >= N
 * are ignored.  Everything else as traj_verify_attn. */
traj_status traj_verify_attn_peers(const void* q, const void* k_cache, const void* v_cache,
                                   const void* k_draft, const void* v_draft,
                                   const int32_t* draft_parent, const uint64_t* draft_peers,
                                   void* out, const traj_attn_shape* shape,
                                   void* workspace, size_t workspace_bytes, void* stream);

/* Peer masks of a joint packing for traj_verify_attn_peers  (Sec. 3.4 "Joint tree
 * construction", App. D).  Per sequence b the drafts [0, n_cur) form the tree of the current
 * block B_t and the drafts [n_cur, n_cur + n_next) the tree of the next block B_{t+1}; each
 * draft of B_t's tree sees the root draft of B_{t+1}'s tree and each draft of B_{t+1}'s tree
 * sees the root draft of B_t's tree:
 *     peers[b, n] = 1 << (n_cur + root_next[b])   for n <  n_cur,
 *     peers[b, n] = 1 << root_cur[b]              for n >= n_cur.
 * root_cur [B] (in [0, n_cur)) and root_next [B] (in [0, n_next)) are int32 device arrays or
 * NULL (root 0); a root outside its tree is taken as 0 and sets TRAJ_DEV_BAD_ROOT.
 * peers: [B, n_cur + n_next] uint64 device output.
 * Limits: B >= 1; n_cur >= 1; n_next >= 1; n_cur + n_next <= 64. */
traj_status traj_joint_peers(int32_t B, int32_t n_cur, int32_t n_next, const int32_t* root_cur,
                             const int32_t* root_next, uint64_t* peers, void* stream);

/* ------------------------------------------------------------------------------------
 * 2. Confidence and top-k candidates  (Sec. 3.2, Eq. 2; "Candidate collection")
 *
 * For each row r of `logits` (rows x vocab, row r starting at logits + r*row_stride
 * elements):
 *     m = max_v l_v,   s = sum_v exp(l_v - m),
 *     idx[r, 0..k-1]  = the k largest entries, larger first; equal values order by the
 *                       lower vocabulary index,
 *     conf[r, j]      = exp(l_idx[r,j] - m) / s          (conf[r,0] is c(x)).
 * Values are compared as stored (bf16 or fp32), the sum and the quotient are fp32.
 * Rows must not contain NaN and must hold at least one finite value.
 * conf: [rows, k] float32, idx: [rows, k] int32 (device).  rows == 0 is a no-op (NULL allowed).
 * Limits: 1 <= k <= 8; k <= vocab; vocab < 2^31; row_stride >= vocab.
 * workspace: may be NULL with workspace_bytes 0; with at least
 * traj_confidence_topk_workspace_size() bytes (16-byte aligned) short batches split each
 * row across several workgroups and merge the partial results.
 * ------------------------------------------------------------------------------------ */
typedef struct {
    int64_t rows, vocab, row_stride;
    int32_t dtype; /* traj_dtype */
} traj_logits_shape;

size_t traj_confidence_topk_workspace_size(const traj_logits_shape* shape, int32_t k);

traj_status traj_confidence_topk(const void* logits, int32_t k, float* conf, int32_t* idx,
                                 const traj_logits_shape* shape,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* traj_confidence_topk for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same kernels and results
 * bit for bit, with the split records of short batches in a fixed scratch array of
 * TRAJ_TOPK_SCRATCH_BYTES that the library holds on each device it runs on until the process
 * ends (its address is looked up on the first call on a device).  Calls no allocating routine.
 * Every call on one device shares that array: calls whose executions overlap on one device
 * (e.g. on two streams) race; calls ordered on one stream do not (nothing in the array needs to
 * start at zero).  A shape whose split records would exceed the array returns TRAJ_E_WORKSPACE
 * (no shape the current plan splits needs more than about 19 KB).  Other arguments, limits and
 * errors as traj_confidence_topk. */
#define TRAJ_TOPK_SCRATCH_BYTES 65536
traj_status traj_confidence_topk_noalloc(const void* logits, int32_t k, float* conf, int32_t* idx,
                                         const traj_logits_shape* shape, void* stream);

/* ------------------------------------------------------------------------------------
 * 3. Acceptance  (Sec. 3.3 "Verification procedure"; Sec. 2.1 threshold decoding;
 *    Sec. 3.1 logit reuse; Alg. 1 phase 1)
 *
 * A block state is an [L] int32 array of token ids with -1 for a masked position.
 * state(-1) = committed[b] with candidates conf0/idx0 (the previous step's output);
 * state(n)  = tokens[b,n]  with candidates conf/idx of draft n's rows.
 * step_tau(s, C, I): if s has no masked position there is no step; otherwise unmask every
 *   masked p with C[p,0] > threshold (strict) with token I[p,0]; if there is none, unmask
 *   only the masked p of largest C[p,0] (smallest p on equal values).
 * Draft c with parent q is consistent when
 *   TRAJ_MODE_EXACT: tokens[c] == step_tau(state(q)) at every position;
 *   TRAJ_MODE_TOP1 : it keeps every unmasked token of state(q), unmasks at least one new
 *                    position, and every new token equals I_q[p,0];
 *   TRAJ_MODE_TOPK : as TOP1 with the new token among I_q[p,0..k-1].
 * Traversal TRAJ_GREEDY walks from the committed state, always taking the lowest-index
 * consistent child; TRAJ_LONGEST takes, among drafts whose whole root path is
 * consistent, the one unmasking the most committed-masked positions (lowest index on
 * ties).  Outputs per sequence:
 *   leaf[b]            accepted draft, -1 if none
 *   on_path[b,n]       1 if draft n lies on the root path of leaf
 *   n_accepted[b]      #positions masked in committed[b] and unmasked in the leaf (0 if none)
 *   out_tokens[b,:]    tokens[b,leaf], or committed[b] when leaf = -1
 *   hi[b,n,p]          1 if tokens[b,n,p] is masked and conf[b,n,p,0] > threshold
 * conf/idx are traj_confidence_topk's outputs for rows ordered (b, n, p): [B,N,L,k].
 * Limits: 1 <= N <= 64; 1 <= L <= 64; 1 <= k <= 8; B >= 1.  All arrays are device arrays.
 * ------------------------------------------------------------------------------------ */
enum { TRAJ_MODE_EXACT = 0, TRAJ_MODE_TOP1 = 1, TRAJ_MODE_TOPK = 2 };
enum { TRAJ_GREEDY = 0, TRAJ_LONGEST = 1 };

typedef struct {
    int32_t B, N, L, k;
    const int32_t* tokens;    /* [B,N,L]  -1 = masked                    */
    const int32_t* parent;    /* [B,N]    -1 = child of committed state  */
    const int32_t* committed; /* [B,L]    committed block state          */
    const float* conf0;       /* [B,L,k]  committed state's confidences  */
    const int32_t* idx0;      /* [B,L,k]  committed state's candidates   */
    int32_t mode;             /* TRAJ_MODE_*                             */
    int32_t traversal;        /* TRAJ_GREEDY or TRAJ_LONGEST             */
} traj_drafts;

typedef struct {
    int32_t* leaf;       /* [B]      */
    uint8_t* on_path;    /* [B,N]    */
    int32_t* n_accepted; /* [B]      */
    int32_t* out_tokens; /* [B,L]    */
    uint8_t* hi;         /* [B,N,L]  */
} traj_accepted;

traj_status traj_accept(const float* conf, const int32_t* idx, const traj_drafts* drafts,
                        float threshold, const traj_accepted* accepted, void* stream);

/* ------------------------------------------------------------------------------------
 * 4. Draft tree construction  (Alg. 1, confidence-stratified trajectory tree; Sec. 3.2
 *    "Tree construction" and "Complexity analysis"; Sec. 3.1 logit reuse)
 *
 * Builds the next step's draft tree of every sequence from the state traj_accept accepted
 * and the candidates the verification pass produced for that state:
 *   s0        = state[b,:]                                   (traj_accept's out_tokens)
 *   (C, I)    = conf[b, leaf[b]], idx[b, leaf[b]]   ([L,k])  when leaf[b] >= 0,
 *               conf0[b], idx0[b]                            when leaf[b] == -1 or leaf == NULL.
 * Phase 1: H = masked p with C[p,0] > threshold (strict), Low = masked p with
 *   C[p,0] <= threshold.  The root is s0 with every p of H set to I[p,0]; when H is not
 *   empty it is node 0 (parent -1), otherwise the root is s0 itself and is not emitted (the
 *   first-level nodes then have parent -1).
 * Phase 2, for levels l = 1 .. depth while Low has an l-th position q_l (Low ranked by
 *   C[p,0], larger first, smaller p on equal values):
 *   l = 1:  children j = 0 .. branch-1 of the root set q_1 to I[q_1, j]     (GenerateTopK);
 *   l > 1:  each kept node of level l-1 gets branch_deep children setting q_l to I[q_l, j],
 *           j = 0 .. branch_deep-1 (GenerateTop1 when branch_deep == 1, the hybrid policy;
 *           2 = the "full top-2" policy of the expansion ablation);
 *   each level keeps its w_l best children by score (PruneByConfidence; generation order on
 *   equal scores, scores compared in fp32), w_l = max(width - l + 1, 1) (hybrid, full == 0)
 *   or width (full == 1).
 *   score = sum of log C over the candidates chosen on the path below the root (root: 0),
 *   accumulated in fp32 in path order.
 *   With H empty, node 0 is one threshold-decoding step of s0 (the top-1 fallback), so an
 *   exact-mode traj_accept of the tree always advances.
 * Outputs (breadth first, each level in kept order; int32 unless stated):
 *   tokens[b,n,:]   block state of node n, -1 = masked            [B, n_max, L]
 *   parent[b,n]     -1 or the generating node's index (< n)       [B, n_max]
 *   n_nodes[b]      number of nodes (0 when s0 has no masked position)  [B]
 *   score[b,n]      float32 path log-confidence (may be NULL)      [B, n_max]
 *   Slots n >= n_nodes[b] hold s0, parent -1 and score -inf: a copy of s0 is never a
 *   consistent child, so the outputs can be verified and accepted as an n_max-draft tree.
 *   conf_next / idx_next (float32 / int32 [B,L,k], may both be NULL): the gathered (C, I),
 *   the committed-state candidates of the next traj_accept call (its conf0 / idx0).
 * Each [k] candidate row must be non-increasing in confidence (as traj_confidence_topk
 * writes it): the first level's pruning keeps candidates 0 .. w_1-1 on that basis.
 * Limits: B >= 1; 1 <= L <= 64; 1 <= k <= 8; 1 <= branch, branch_deep <= k; width >= 1; depth >= 0;
 *   n_prev >= 0 (drafts per sequence in conf / idx; both may be NULL when n_prev == 0 or
 *   leaf == NULL); traj_tree_max_nodes(shape) <= n_max <= 64.
 *   A leaf[b] outside [-1, n_prev) is taken as -1 and sets TRAJ_DEV_BAD_LEAF.
 * ------------------------------------------------------------------------------------ */
typedef struct {
    int32_t B, L, k;
    int32_t n_prev;               /* drafts per sequence in conf / idx                 */
    int32_t width, depth, branch; /* W, D and the candidates tried at the first level  */
    int32_t full;                 /* 0 hybrid level widths, 1 full (width per level)   */
    int32_t n_max;                /* node slots per sequence in the outputs            */
    int32_t branch_deep;          /* children per node below the first level, 1..k     */
} traj_tree_shape;

/* Largest node count the shape's tree can reach (1 + sum over levels l <= min(depth, L) of
 * c_l, c_1 = min(branch, w_1), c_l = min(w_l, c_{l-1} * branch_deep)); -1 when the shape is
 * invalid. */
int32_t traj_tree_max_nodes(const traj_tree_shape* shape);

traj_status traj_build_tree(const int32_t* state, const int32_t* leaf, const float* conf,
                            const int32_t* idx, const float* conf0, const int32_t* idx0,
                            const traj_tree_shape* shape, float threshold, int32_t* tokens,
                            int32_t* parent, int32_t* n_nodes, float* score, float* conf_next,
                            int32_t* idx_next, void* stream);

/* ------------------------------------------------------------------------------------
 * 5. Inter-block speculation trigger  (Sec. 3.4 "Trigger condition", App. D)
 *
 * For every sequence b, with the states and candidates of two consecutive blocks packed as
 * 2L positions (B_t at 0..L-1, B_{t+1} at L..2L-1; one verification pass whose drafts cover
 * both blocks produces them):
 *   c_cur[b]  = max of conf[b,p,0] over masked p < L           (0 when none is masked)
 *   c_next[b] = max of conf[b,p,0] over masked L <= p < 2L     (0 when none is masked)
 *   trigger[b] = 1 iff B_{t+1} has a masked position and (c_next > c_cur or c_next > threshold),
 * in fp32, strict comparisons.
 * state [B, 2L] int32 (-1 = masked), conf [B, 2L, k] float32 (traj_confidence_topk's rows),
 * trigger [B] uint8, c_cur / c_next [B] float32 (each may be NULL).
 * Limits: B >= 1; 1 <= L <= 64; 1 <= k <= 8.
 * ------------------------------------------------------------------------------------ */
traj_status traj_interblock_trigger(const int32_t* state, const float* conf, int32_t B, int32_t L,
                                    int32_t k, float threshold, uint8_t* trigger, float* c_cur,
                                    float* c_next, void* stream);

/* ------------------------------------------------------------------------------------
 * 6. Verification layer  (Sec. 3.2 "Complexity analysis": the drafts go through one
 *    concatenated forward pass; Sec. 3.3: with the trajectory mask; App. A: dual cache)
 *
 * One pre-norm decoder layer of the 8B-shaped diffusion LMs over the packed draft tokens,
 * updating their residual stream x in place:
 *   xn = RMSNorm(x) * attn_norm;   [q | k | v] = xn @ w_qkv;   RoPE on q and k;
 *   x += traj_verify_attn(q, k_cache, v_cache, k, v, draft_parent) @ w_o;
 *   xn = RMSNorm(x) * mlp_norm;    [g | u] = xn @ w_gate_up;   x += (silu(g) * u) @ w_down.
 * RMSNorm: x / sqrt(mean(x^2) + rms_eps).  RoPE: pairs (d, d + D/2) of each q / k head rotate
 * by pos * rope_theta^(-2d/D), pos = pos0[b] + p for block position p of every draft (the drafts
 * are alternative states of the same block); the cache K is expected with RoPE applied.
 * Every intermediate is rounded to bf16 (the activations' storage type), arithmetic is fp32;
 * the projections are the library's own bf16 MFMA GEMM (fp32 accumulation, the residual
 * additions fused into the O and down projections).
 * Layouts (bf16, row-major): x [B,N,L,hidden]; attn_norm, mlp_norm [hidden];
 *   w_qkv [hidden, (Hq + 2 Hkv) D]; w_o [Hq D, hidden]; w_gate_up [hidden, 2 inter] (gate then
 *   up); w_down [inter, hidden]; k_cache / v_cache and draft_parent as traj_verify_attn;
 *   pos0 [B] int32 (NULL = 0).  shape is the attention shape of the call (scale included).
 * workspace: at least traj_verify_layer_workspace_size() bytes, 256-byte aligned (the
 * intermediates: normed x, q/k/v, attention output, gate/up, activation; and the split-K
 * partial products of the projections for few-row shapes, as traj_linear).
 * Limits: those of traj_verify_attn; hidden == Hq * D; hidden % 8 == 0; inter % 8 == 0.
 * ------------------------------------------------------------------------------------ */
typedef struct {
    int32_t hidden, inter;
    float rms_eps, rope_theta;
} traj_layer_dims;

typedef struct {
    const void* attn_norm;
    const void* w_qkv;
    const void* w_o;
    const void* mlp_norm;
    const void* w_gate_up;
    const void* w_down;
} traj_layer_weights;

size_t traj_verify_layer_workspace_size(const traj_attn_shape* shape, const traj_layer_dims* dims);

traj_status traj_verify_layer(void* x, const traj_layer_weights* weights, const traj_layer_dims* dims,
                              const void* k_cache, const void* v_cache, const int32_t* draft_parent,
                              const int32_t* pos0, const traj_attn_shape* shape, void* workspace,
                              size_t workspace_bytes, void* stream);

/* Dual-cache refresh at a block boundary (App. A: the prefix / suffix K and V the verification
 * layer reads during a block's speculation are computed once per block, over the whole
 * sequence).  One decoder layer, the same as traj_verify_layer's, over B whole sequences of
 * T = S + L tokens (prefix | current block | suffix) with bidirectional attention over all T
 * tokens of the sequence, updating x in place.  The layer's rotated K and its V of every
 * position outside the block [block_start[b], block_start[b] + L) are written to
 * k_cache / v_cache (prefix rows, then suffix rows): the cache traj_verify_layer takes.
 * Positions: token t of a sequence sits at position t (block tokens at block_start + p, the
 * positions traj_verify_layer gives the drafts with pos0 = block_start).
 * Layouts (bf16): x [B, T, hidden]; k_cache / v_cache [B, S, Hkv, D] (written); block_start [B]
 * int32 device array in [0, S] (a value outside is clamped and sets TRAJ_DEV_BAD_BLOCK).
 * Weights, dims, rounding and limits as traj_verify_layer (shape->scale 0 = 1/sqrt(D)); one
 * sequence's T K / V rows must stay below 2 GiB.  x, the caches and the workspace must not overlap.
 * workspace: at least traj_refresh_layer_workspace_size() bytes, 256-byte aligned. */
typedef struct {
    int32_t B, S, L, Hq, Hkv, D;
    float scale;
} traj_refresh_shape;

size_t traj_refresh_layer_workspace_size(const traj_refresh_shape* shape, const traj_layer_dims* dims);

traj_status traj_refresh_layer(void* x, const traj_layer_weights* weights, const traj_layer_dims* dims,
                               const int32_t* block_start, void* k_cache, void* v_cache,
                               const traj_refresh_shape* shape, void* workspace, size_t workspace_bytes,
                               void* stream);

/* The layer's projection GEMM on its own (also the LM head of the verification forward,
 * whose logits traj_confidence_topk reads; Sec. 3.2 "Complexity analysis"):
 *   y[M,N] = x[M,K] @ w[K,N]            (accumulate == 0)
 *   y[M,N] = x[M,K] @ w[K,N] + y[M,N]   (accumulate != 0; y is read, then overwritten)
 * bf16 row-major operands, fp32 accumulation, each result rounded once to bf16 (nearest even).
 * Limits: K and N multiples of 8 (>= 8), M >= 0 (0 = no-op) and below 2^31 - 256, pointers
 * 16-byte aligned; y must not overlap x or w.  The kernels address operands through 32-bit
 * buffer offsets: K <= 2^22 and N <= 2^24, else TRAJ_E_UNSUPPORTED.  Nothing is allocated.
 * workspace (optional, may be NULL): shapes whose 128 x 128 tiles leave CUs idle (few rows:
 * one or a few sequences' drafts) split K over several workgroups when given at least
 * traj_linear_workspace_size(M, K, N) bytes, 16-byte aligned, for the fp32 partial products
 * (a size of 0 means the shape is never split); with NULL the call runs unsplit.  A non-NULL
 * workspace that is too small or misaligned is TRAJ_E_WORKSPACE; it must not overlap x, w or y.
 * Errors: TRAJ_E_SHAPE (sizes, alignment), TRAJ_E_UNSUPPORTED, TRAJ_E_NULL, TRAJ_E_WORKSPACE,
 * TRAJ_E_HIP (launch). */
size_t traj_linear_workspace_size(int64_t M, int64_t K, int64_t N);

traj_status traj_linear(const void* x, const void* w, void* y, int64_t M, int64_t K, int64_t N, int32_t accumulate,
                        void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------------------
 * Utilities
 * ------------------------------------------------------------------------------------ */
/* Static, NUL-terminated description of a status code (never NULL). */
const char* traj_status_string(int32_t status);
/* Static version string of the library: "libtrajspec <version> gfx950 sources <sha256>", the
 * digest of the sources and compiler flags it was built from ("unstamped" when built without
 * the package's build script). */
const char* traj_version(void);
/* Synchronises `stream`, copies the current device's status word (TRAJ_DEV_* bits) to
 * *host_flags and, if reset != 0, clears it.  Returns TRAJ_E_HIP on a runtime error. */
traj_status traj_get_device_status(int32_t* host_flags, int32_t reset, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* TRAJ_SPEC_H */
