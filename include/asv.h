/*
 * asv.h — C ABI of libasv, the MI355X (gfx950) verification path of AdaptiveSpec
 * ("Margins, Not Windows: Training-Free Per-Step Lossy Speculative Decoding").
 *
 * One call, asv_verify(), scores every draft-tree node of a batch with the target LM head and
 * applies the paper's margin rule (Sec. 3.2, Eq. (1)): a drafted token d whose target
 * probability ratio p(d) / p(top1) reaches the threshold kappa (here `tau`) is accepted even
 * when it is not the target's top-1, i.e. z_d - z_max >= ln(tau). It then walks each request's
 * tree, returns the accepted path and the bonus token, and updates the per-request signals the
 * adaptive tree policy reads (Sec. 3.3: draft top-1 confidence of Eq. (2) and the rolling
 * acceptance rate with its circuit breaker).
 *
 * Around it: asv_draft_step / asv_draft_prune build the next draft tree from the draft model's
 * LM head (Sec. 2, "Draft": topk-way branching, pruning to ndt tokens) in the shape the policy
 * state selects; asv_tree_meta gives the target forward its positions and tree-attention mask;
 * asv_commit gathers what a verification step commits.
 *
 * Conventions shared by every entry point:
 *   - Every array argument is DEVICE memory owned by the caller (e.g. a torch tensor's
 *     data_ptr()). The library never allocates, frees or keeps a pointer after a call returns.
 *   - `stream` is a hipStream_t (NULL = the default stream). Work is enqueued asynchronously on
 *     it with no host synchronisation; outputs are valid once the caller synchronises it.
 *   - Return value: ASV_OK, or a negative ASV_E* code detected on the host before anything is
 *     enqueued (outputs are then untouched). Problems that only the data can show are reported
 *     per request in `req_status` (ASV_RS_* bits) and never fault the GPU.
 *   - bf16 values are passed as raw 16-bit patterns (uint16_t), row-major, rows contiguous.
 *   - Calls that share one workspace or one state array must be ordered on one stream.
 */
#ifndef ASV_H_
#define ASV_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ASV_VERSION 160          /* 1.6.0 */

/* Return codes. */
#define ASV_OK          0
#define ASV_EINVAL     -1        /* bad size, null or misaligned pointer, bad parameter */
#define ASV_EWORKSPACE -2        /* workspace smaller than asv_workspace_bytes() or misaligned */
#define ASV_EHIP       -3        /* a HIP runtime call or kernel launch failed */
#define ASV_ESCRATCH   -4        /* asv_verify_noalloc: the sizes need more workspace than the
                                    library's static scratch holds */

/* req_status bits, set on the device for request b. A request with any bit set gets
 * accepted_len = 0, bonus_token = -1, draft_conf = NaN and its state left unchanged; its path
 * entries and accept flags are cleared, except under ASV_RS_BAD_OFFSETS, where the request's
 * rows are unknown and neither is written. Row statistics (row_max, row_lse, row_argmax,
 * drafted_logit) are produced for all N rows in every case. */
#define ASV_RS_BAD_ROOT    1     /* parent[req_offsets[b]] != -1 */
#define ASV_RS_BAD_PARENT  2     /* a non-root c has parent outside [req_offsets[b], c) */
#define ASV_RS_BAD_TOKEN   4     /* a non-root draft_tok outside [0, V) */
#define ASV_RS_BAD_OFFSETS 16    /* the offsets array is malformed: not strictly
                                    increasing, req_offsets[0] != 0 or req_offsets[B] != N.
                                    Set on every request of the batch. */
#define ASV_RS_BAD_TAU     32    /* tau[b] outside [0, 1] or NaN */
#define ASV_RS_MASK_SMALL  64    /* asv_tree_meta: the request has more than 32 * mask_words
                                    nodes; its positions are written, its mask rows are not */
#define ASV_RS_BAD_PATH    128   /* asv_commit: accepted_len[b] outside [0, n_b - 1] or an
                                    accepted_path entry that is not a node of request b */

#define ASV_HIST_WINDOW 16

/* Per-request policy state (Sec. 3.3), caller-owned device memory, 112 bytes, in/out.
 * Initialise with asv_state_init(); copy the bytes to checkpoint or resume. */
typedef struct asv_req_state {
  float   rar;                      /* rolling acceptance rate, an EMA of the accept fraction */
  float   hist[ASV_HIST_WINDOW];    /* ring of the last accept fractions */
  int32_t hist_head;                /* next ring slot to write */
  int32_t hist_count;               /* filled ring slots, <= 16 */
  int32_t zero_streak;              /* consecutive steps that accepted no drafted token */
  int32_t breaker;                  /* 1 when this step tripped the circuit breaker */
  int32_t steps;                    /* verify steps seen */
  float   hist_mean;                /* mean of the filled ring slots (rar0 when empty) */
  float   draft_conf;               /* last p_draft(top1) of Eq. (2), when draft logits given */
  float   dcs;                      /* Draft Confidence Score of Eq. (2),
                                       min(1, draft_conf * rar / dcs_divisor) */
  int32_t shape[3];                 /* (nsteps, topk, ndt) the score selects for the next draft
                                       tree; the starting configuration after a breaker trip */
} asv_req_state;

/* Policy parameters (Sec. 3.3 and Appendix B). */
typedef struct asv_params {
  float   alpha;           /* EMA weight of the newest observation, in (0, 1]; paper: 0.3 */
  float   rar0;            /* RAR before the first step and after a breaker trip; 1.0 */
  int32_t breaker_n;       /* zero-accept steps that trip the breaker, >= 1; paper: 5 */
  int32_t max_promotions;  /* mismatches one walk may promote; -1 = no limit, 1 = only the
                              first mismatch position */
  float   temperature;     /* T > 0 of the margin exp((z_d - z_max) / T) >= kappa, the target
                              distribution taken as softmax(z / T); 1 is Eq. (1) */
  float   dcs_divisor;     /* d of Eq. (2): the score saturates once p_draft * RAR reaches d,
                              > 0; paper: 0.5 */
  int32_t shape_lo[3];     /* (nsteps, topk, ndt) at score 0, each >= 1; paper: (3, 4, 4) */
  int32_t shape_hi[3];     /* the same at score 1; paper: (7, 1, 8) */
  int32_t shape_start[3];  /* the starting configuration: the shape before the first step and
                              after a breaker trip; (3, 4, 4) here */
} asv_params;

/* Arguments of asv_verify. Shapes use B requests and N tree rows in total. Request b owns the
 * contiguous rows [req_offsets[b], req_offsets[b+1]); its first row is the root (the last
 * committed token, not drafted, parent -1). Every other row c is a drafted node whose token
 * draft_tok[c] is judged by the target distribution predicted at its parent's row. */
typedef struct asv_verify_args {
  int32_t B, N, H, V;             /* host ints: B >= 0, N >= B (N == 0 iff B == 0),
                                     H > 0 with H % 64 == 0 and H <= 2^20, V > 0,
                                     N, V < 2^30 and ceil(V / 256) * ceil(N / 64) < 2^31
                                     (the LM-head kernel's largest workgroup count) */
  const uint16_t *hidden;         /* [N][H] bf16 final hidden states, 16-byte aligned */
  const uint16_t *w_lm;           /* [V][H] bf16 LM-head weight, or its packed copy (see
                                     w_lm_layout), 16-byte aligned */
  const int32_t  *draft_tok;      /* [N] drafted token ids; root entries ignored */
  const int32_t  *parent;         /* [N] global row id of each node's parent; -1 at roots;
                                     req_offsets[b] <= parent[c] < c inside request b */
  const int32_t  *req_offsets;    /* [B+1] row offsets, req_offsets[0] = 0, [B] = N */
  const float    *tau;            /* [B] margin threshold kappa in [0, 1]; 0 accepts all,
                                     1 is strict token match */
  const float    *draft_logits;   /* [N][V] fp32 draft-model logits, or NULL. Only each
                                     request's root row is read (Eq. (2)). */
  /* outputs, all [N] unless noted */
  float   *row_max;               /* max_v z_n[v] of row n */
  float   *row_lse;               /* log sum_v exp(z_n[v]) of row n */
  int32_t *row_argmax;            /* lowest v attaining row_max */
  float   *drafted_logit;         /* z_{parent(c)}[draft_tok[c]]; roots: unspecified */
  uint8_t *accept;                /* Eq. (1) verdict of each node (1 = accept); roots 1 */
  int32_t *accepted_len;          /* [B] accepted drafted tokens (root and bonus excluded) */
  int32_t *bonus_token;           /* [B] target argmax at the last accepted node */
  int32_t *accepted_path;         /* [N] request b's accepted node ids (global rows, root
                                     excluded) at [req_offsets[b], +accepted_len[b]); the
                                     rest of its segment is -1 */
  float   *draft_conf;            /* [B] p_draft(top1) of each root row, or NULL */
  asv_req_state *state;           /* [B] in/out policy state, or NULL to skip the update */
  int32_t *req_status;            /* [B] ASV_RS_* bits, 0 when the request was well formed */
  asv_params params;
  int32_t w_lm_layout;            /* ASV_W_ROW_MAJOR: w_lm is [V][H] as above.
                                     ASV_W_PACKED: w_lm is the output of asv_pack_lm_head for
                                     this V and H. Both give bit-identical results. Any other
                                     value, or ASV_W_PACKED for sizes asv_packed_lm_head_bytes
                                     rejects: ASV_EINVAL */
} asv_verify_args;

/* Layouts of the LM-head weight that asv_verify reads. */
#define ASV_W_ROW_MAJOR 0
#define ASV_W_PACKED    1

/* The packed layout: the [V][H] weight cut into S = ceil(V / 256) slabs of 256 vocabulary rows
 * and K = H / 64 column blocks of 64; block (slab s, columns k) is a [256][64] tile, and the
 * tiles are stored column block major:
 *   packed[((k * S + s) * 256 + r) * 64 + c] = w[256 s + r][64 k + c],
 * zero where 256 s + r >= V. It holds S * 256 * H bf16 values. Each 64-deep step of the
 * LM-head kernel reads one [256][64] tile per slab, and the slabs advance through K together,
 * so at every step the whole launch reads one contiguous window instead of 256 runs of 128
 * bytes per slab, each 2 H bytes apart. The rate of those strided runs depends on where the
 * weight sits in physical memory; the contiguous window streams at the same rate wherever it
 * sits. The logits are summed in the same order from the same values. Pack once when the
 * weights are loaded: the LM-head weight is a constant of the model. */

/* Bytes of the packed copy of a [V][H] LM-head weight. Returns ASV_EINVAL for V <= 0, for an
 * H that asv_verify would reject, or for a packed copy of 4 GiB or more (S * H / 64 >= 2^17):
 * pass such weights row-major. */
int asv_packed_lm_head_bytes(int32_t V, int32_t H, uint64_t *bytes);

/* Write the packed copy of the [V][H] bf16 weight w (16-byte aligned) into `packed`
 * (16-byte aligned, packed_bytes >= asv_packed_lm_head_bytes(V, H), not overlapping w).
 * Enqueued on `stream`. Returns ASV_EINVAL for bad sizes, null, misaligned or overlapping
 * pointers, a packed_bytes too small; ASV_EHIP if the launch fails. */
int asv_pack_lm_head(const uint16_t *w, int32_t V, int32_t H, uint16_t *packed,
                     uint64_t packed_bytes, void *stream);

/* ---- Draft side (Sec. 2, "Draft"): the draft model runs nsteps forwards, every frontier node
 * branches topk ways, and the tree is pruned to a verification budget of ndt tokens (ndt counts
 * the root). The tree grows as in EAGLE-2 (the drafter the paper adopts, EAGLE-3, grows its tree
 * this way): a node's score is the float32 sum of the draft log-probabilities along its path;
 * each step appends all frontier x topk children to the node pool (frontier slot major, child
 * rank minor) and keeps the topk best as the next frontier (best first, the earlier candidate on
 * equal scores); pruning keeps the root and the ndt - 1 best pool nodes (the earlier pool entry
 * on equal scores) in pool order, so parents precede children. */

#define ASV_TOPK_MAX 4           /* largest topk of a draft tree = width of the draft top-k */
#define ASV_POOL_MAX 256         /* drafted nodes one tree can hold: topk + (nsteps-1) topk^2 */

/* asv_draft_tree.status and asv_draft_prune req_status bits. */
#define ASV_DS_BAD_SHAPE 1       /* shape outside nsteps >= 1, 1 <= topk <= 4, ndt >= 1, or a
                                    pool larger than ASV_POOL_MAX: the tree stays root-only */
#define ASV_DS_OVERFLOW  2       /* asv_draft_prune: the request's rows end past n_cap; none of
                                    them is written */

/* One request's draft tree while it grows. Caller-owned device memory, 3136 bytes, written by
 * asv_draft_step (initialised at step 0) and read by asv_draft_prune. */
typedef struct asv_draft_tree {
  int32_t nsteps, topk, ndt;        /* the shape the tree grows to, fixed at step 0 */
  int32_t steps;                    /* draft steps applied so far */
  int32_t n_pool;                   /* drafted nodes in the pool */
  int32_t n_front;                  /* frontier slots; 1 (the root) before the first step */
  int32_t status;                   /* ASV_DS_* bits, 0 when the shape was valid */
  int32_t reserved;
  int32_t front[ASV_TOPK_MAX];      /* pool index of each frontier slot, best first; -1 = root */
  float   front_score[ASV_TOPK_MAX];
  int32_t tok[ASV_POOL_MAX];        /* drafted token of each pool node (a target id) */
  int32_t par[ASV_POOL_MAX];        /* pool index of its parent, -1 for a child of the root */
  float   score[ASV_POOL_MAX];       /* sum of the float32 log-probabilities along its path */
} asv_draft_tree;

/* Arguments of asv_draft_step. Draft rows use a fixed stride of ASV_TOPK_MAX per request: row
 * 4b + j holds the draft model's final hidden state for frontier slot j of request b (at step 0
 * only slot 0, the root, is read by the tree update). Rows of unused slots are computed like any
 * other row and then ignored, so they may hold anything. */
typedef struct asv_draft_args {
  int32_t B, H, V;                /* host ints: B >= 0, H > 0 with H % 64 == 0,
                                     4 <= V < 2^30, 8 B H < 2^31, and the draft LM head's
                                     workgroup count (slabs x row tiles) below 2^31 */
  int32_t step;                   /* host int: 0 (re)starts every tree from its shape */
  const uint16_t *hidden;         /* [4B][H] bf16 draft hidden states, 16-byte aligned */
  const uint16_t *w_draft;        /* [V][H] bf16 draft LM-head weight, 16-byte aligned */
  const int32_t  *vocab_map;      /* [V] draft id -> target id, or NULL for the identity */
  const asv_req_state *state;     /* [B]: at step 0 tree b takes state[b].shape; or NULL */
  int32_t shape[3];               /* (nsteps, topk, ndt) for every tree when state is NULL */
  asv_draft_tree *tree;           /* [B] in/out */
  /* outputs */
  int32_t *topk_id;               /* [4B][4] the 4 most probable tokens of each row, best first
                                     (lowest draft id on equal logits; a non-number logit
                                     counts as -inf), mapped through vocab_map */
  float   *topk_logp;             /* [4B][4] their log-probabilities z - lse (non-number: -inf) */
  float   *row_lse;               /* [4B] log sum_v exp(z[v]) over the draft vocabulary */
  int32_t *front_tok;             /* [B][4] token of each new frontier slot (the next draft
                                     forward's inputs); -1 for slots past the frontier and for
                                     trees that are done or invalid */
  float   *draft_conf;            /* [B] or NULL; at step 0, p_draft(top1) = exp(best log-prob of
                                     the root row), the confidence Eq. (2) reads */
  int32_t w_draft_layout;         /* ASV_W_ROW_MAJOR: w_draft is [V][H] as above.
                                     ASV_W_PACKED: w_draft is the output of asv_pack_draft_head
                                     for this V and H. Both give bit-identical results. Any
                                     other value, or ASV_W_PACKED for sizes
                                     asv_packed_draft_head_bytes rejects: ASV_EINVAL */
} asv_draft_args;

/* Workspace asv_draft_step needs (per-vocabulary-slab top-4 records); 256-byte aligned, no
 * initialisation needed. Returns ASV_EINVAL for sizes asv_draft_step would reject. */
int asv_draft_workspace_bytes(int32_t B, int32_t H, int32_t V, uint64_t *bytes);

/* The packed draft LM-head weight: the same idea as asv_pack_lm_head with [64][64] tiles, since
 * the draft LM-head kernel reads slabs of 64 or 128 vocabulary rows. With Vp = V rounded up to
 * a multiple of 128 and T = Vp / 64 tiles per 64-column block:
 *   packed[((k * T + s) * 64 + r) * 64 + c] = w[64 s + r][64 k + c], zero where 64 s + r >= V.
 * It holds Vp * H bf16 values. asv_packed_draft_head_bytes returns ASV_EINVAL for sizes
 * asv_draft_step would reject or a copy of 4 GiB or more; asv_pack_draft_head takes the same
 * arguments and gives the same errors as asv_pack_lm_head. */
int asv_packed_draft_head_bytes(int32_t V, int32_t H, uint64_t *bytes);
int asv_pack_draft_head(const uint16_t *w, int32_t V, int32_t H, uint16_t *packed,
                        uint64_t packed_bytes, void *stream);

/* One draft step for a batch (Sec. 2, "Draft"): the draft LM head over all 4B rows (bf16 inputs,
 * fp32 accumulation) reduced on the fly to each row's top-4 and log-sum-exp (the [4B][V] logits
 * never reach memory), then one growth step of every tree that has not taken its nsteps steps.
 * Returns ASV_EINVAL for bad sizes, null or misaligned pointers or (state NULL) a bad shape,
 * ASV_EWORKSPACE, or ASV_EHIP. A bad shape read from state marks that tree ASV_DS_BAD_SHAPE. */
int asv_draft_step(const asv_draft_args *args, void *workspace, uint64_t workspace_bytes,
                   void *stream);

/* Prune every tree to its verification budget and lay the batch out as asv_verify reads it:
 * request b gets n_b = 1 + min(ndt - 1, n_pool) rows at [req_offsets[b], req_offsets[b+1]),
 * the root first (parent -1, draft_tok = root_tok[b], or -1 when root_tok is NULL), then the
 * kept pool nodes in pool order with global parent ids. An invalid tree gives n_b = 1.
 * tree: [B]; root_tok: [B] or NULL; parent, draft_tok: [n_cap]; req_offsets: [B+1] (always
 * written, also past n_cap); req_status: [B] ASV_DS_* bits. Returns ASV_EINVAL for B < 0,
 * n_cap < 0 or null outputs, ASV_EHIP if a launch fails. */
int asv_draft_prune(const asv_draft_tree *tree, int32_t B, const int32_t *root_tok,
                    int32_t n_cap, int32_t *parent, int32_t *draft_tok, int32_t *req_offsets,
                    int32_t *req_status, void *stream);

/* ---- Around the target forward. */

/* Tree-attention metadata (Sec. 1, Sec. 2: the target scores the whole tree in one forward).
 * For node c of request b: pos[c] = pos_base[b] + depth(c) (pos_base NULL: 0), depth being the
 * number of parent links to the root; mask row c, mask_words 32-bit words at mask + c *
 * mask_words, has bit (j - req_offsets[b]) set iff node j is c or an ancestor of c (bit k of
 * word k / 32 at position k % 32). pos or mask may be NULL to skip them. Requests whose
 * offsets or parents are malformed (ASV_RS_BAD_OFFSETS, ASV_RS_BAD_ROOT, ASV_RS_BAD_PARENT)
 * get neither; a request with more than 32 * mask_words nodes gets ASV_RS_MASK_SMALL and its
 * positions only. req_status: [B]. Returns ASV_EINVAL for bad sizes or null arguments. */
int asv_tree_meta(const int32_t *parent, const int32_t *req_offsets, int32_t B, int32_t N,
                  const int32_t *pos_base, int32_t mask_words, int32_t *pos, uint32_t *mask,
                  int32_t *req_status, void *stream);

/* Arguments of asv_commit: what one verification step commits (Sec. 2, "Verify"). */
typedef struct asv_commit_args {
  int32_t B, N;                   /* host ints, as in asv_verify */
  const int32_t *req_offsets;     /* [B+1] the verified batch's offsets */
  const int32_t *draft_tok;       /* [N] */
  const int32_t *accepted_len;    /* [B] asv_verify outputs */
  const int32_t *accepted_path;   /* [N] */
  const int32_t *bonus_token;     /* [B] */
  int32_t *commit_off;            /* [B+1] prefix sums of accepted_len + 1 */
  int32_t *commit_tok;            /* [N] request b's accepted drafted tokens then its bonus,
                                     at [commit_off[b], commit_off[b+1]) */
  int32_t *commit_row;            /* [N] the rows that stay valid: the root, then the accepted
                                     nodes (global ids) */
  const void *row_src;            /* [N][row_bytes] per-node data to keep (hidden states, KV
                                     slot ids), or NULL */
  void    *row_dst;               /* [N][row_bytes]: row_src[commit_row[i]] lands at row i */
  int64_t row_bytes;              /* > 0 and a multiple of 4 when row_src is given */
  int32_t *req_status;            /* [B] ASV_RS_BAD_OFFSETS / ASV_RS_BAD_PATH bits */
} asv_commit_args;

/* Commit one verification step. A request with ASV_RS_BAD_PATH commits only its root row and
 * bonus (length 0); entries that would land at index >= N are not written. Returns ASV_EINVAL
 * for bad sizes, null or misaligned pointers, ASV_EHIP if a launch fails. */
int asv_commit(const asv_commit_args *args, void *stream);

/* ---- For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): asv_verify with its workspace taken from a
 * scratch array that the library holds in device memory, ASV_STATIC_SCRATCH_BYTES per GPU it
 * runs on, from its first use on that GPU until the process ends. The caller still passes
 * every input and output through `args`, as for asv_verify.
 *
 * The call allocates nothing and frees nothing. Every call on one GPU shares that GPU's scratch
 * and leaves its contents behind; nothing in it needs to start at zero (the kernels clear their
 * own counters). Calls that may overlap on one GPU (several host threads, or several streams
 * without ordering between them) race on the scratch and give undefined results: order them
 * on one stream. Returns ASV_ESCRATCH, before anything is enqueued, when
 * asv_workspace_bytes(B, N, H, V) exceeds ASV_STATIC_SCRATCH_BYTES (for example more than
 * about 4500 rows at V = 151936); ASV_EHIP if the scratch's device address cannot be obtained
 * (asv_last_error() names the call); otherwise asv_verify's results and errors. */
#define ASV_STATIC_SCRATCH_BYTES (32u << 20)
int asv_verify_noalloc(const asv_verify_args *args, void *stream);

/* ASV_VERSION of the loaded library. */
int asv_version(void);

/* Static, human-readable text for an ASV_* return code. */
const char *asv_status_string(int code);

/* Details of the most recent ASV_EHIP or ASV_ESCRATCH failure on the calling host thread (the
 * failing launch or runtime call and the HIP error text, or the bytes needed); "" if none.
 * Valid until the next failing call on this thread. */
const char *asv_last_error(void);

/* Device workspace that asv_verify needs for these sizes (partial per-vocab-slab records of
 * the LM-head kernel and draft-confidence partials). Writes the byte count to *bytes. The
 * workspace must be 256-byte aligned; its contents need no initialisation and are
 * overwritten by every call. Returns ASV_EINVAL for sizes asv_verify would reject. */
int asv_workspace_bytes(int32_t B, int32_t N, int32_t H, int32_t V, uint64_t *bytes);

/* Tree shape for the next draft (Sec. 3.3, Eq. (2)). For each request b: if conf is not NULL,
 * state[b].draft_conf = conf[b] (a fresh p_draft(top1), e.g. from the next step's first draft
 * forward); then state[b].dcs = min(1, draft_conf * rar / d) and state[b].shape = each member
 * of the triplet moved linearly from shape_lo (score 0) to shape_hi (score 1), rounded to the
 * nearest integer with halves down, or shape_start when state[b].breaker is set. The score is
 * computed in float32 with one rounding per operation. asv_verify applies the same rule after
 * its history update, with the step's own draft confidence. conf: [B] device floats or NULL;
 * state: [B] device, in/out. Enqueued on `stream`. Returns ASV_EINVAL for B < 0, a NULL state
 * with B > 0 or invalid parameters, ASV_EHIP if the launch fails. */
int asv_tree_policy(const float *conf, asv_req_state *state, int32_t B, const asv_params *p,
                    void *stream);

/* Fill state[0..B) with the initial policy state for params *p (rar = hist_mean = rar0,
 * empty ring, zero counters, dcs 0, shape = shape_start) on `stream`. */
int asv_state_init(asv_req_state *state, int32_t B, const asv_params *p, void *stream);

/* ---- Measurement and tuning. Not needed to use the library: the product entry points
 * (asv_verify, asv_draft_step) are these calls with a NULL asv_tuning. */

typedef struct asv_tuning {
  void   *begin_event;            /* optional hipEvent_t (created by the caller) set to the
                                     start time of the LM-head kernel's first launch (K1 of
                                     asv_verify, the draft LM head of asv_draft_step), taken from
                                     the dispatch itself (hipExtLaunchKernel), or NULL */
  void   *end_event;              /* optional hipEvent_t set to the end time of its last
                                     launch, or NULL; hipEventElapsedTime(begin, end) is then
                                     the kernel's own time, without event-record packets */
  int32_t tile_rows;              /* asv_verify only: tree rows per LM-head tile. 0 lets the
                                     library pick it from N, V and the device's compute-unit
                                     count; 64, 128, 192 or 256 force that tile (every tile
                                     gives the same results). Any other value, or a nonzero
                                     value for asv_draft_step: ASV_EINVAL */
} asv_tuning;

/* asv_verify / asv_draft_step with measurement and tuning controls; `tuning` may be NULL.
 * Same arguments, results and errors as the product calls; an event that cannot be recorded
 * returns ASV_EHIP. */
int asv_verify_tuned(const asv_verify_args *args, const asv_tuning *tuning, void *workspace,
                     uint64_t workspace_bytes, void *stream);

/* One launch of the LM-head kernel of asv_verify (see asv_k1_plan). */
typedef struct asv_k1_launch {
  int32_t tile_rows;              /* tree rows per workgroup tile: 64, 128, 192 or 256 */
  int32_t slab0;                  /* first vocabulary slab (256 ids each) of the launch */
  int32_t n_slabs;                /* slabs it covers */
  int32_t row_tiles;              /* tiles along the tree rows: ceil(N / tile_rows) */
  int32_t k_loop;                 /* 0 burst ring, 1 one-slot ring, 2 two-slot spread loop,
                                     3 three-slot spread loop */
  int32_t stream_w;               /* 1: the weight is copied with the non-temporal hint */
  int32_t blk_slabs, blk_rows;    /* tile order: blocks of blk_slabs slabs x blk_rows row
                                     tiles, or 0 and 0 for the slab-major order */
} asv_k1_launch;

/* The LM-head launches asv_verify (asv_verify_tuned with tile_rows forced, 0 = the library's
 * choice) enqueues for N tree rows and V vocabulary ids on a GPU with `cus` compute units:
 * fills launches[0 .. *n_launches), at most two, in launch order. Host computation only; no
 * GPU call. ASV_EINVAL for N < 1, V < 1, N and V beyond asv_verify_args' bound, cus < 1, a
 * tile_rows asv_tuning rejects or null pointers. */
int asv_k1_plan(int32_t N, int32_t V, int32_t cus, int32_t tile_rows, asv_k1_launch *launches,
                int32_t *n_launches);
int asv_draft_step_tuned(const asv_draft_args *args, const asv_tuning *tuning, void *workspace,
                         uint64_t workspace_bytes, void *stream);

/* One verification step for a batch (Sec. 3.2, Eq. (1); Sec. 3.3, Eq. (2)):
 *   1. logits of every row against every vocabulary entry (bf16 inputs, fp32 accumulation),
 *      reduced on the fly to row_max / row_lse / row_argmax and the drafted logits — the
 *      [N][V] logits matrix is never written to memory;
 *   2. accept[c] = (draft_tok[c] == row_argmax[p]) || tau == 0 ||
 *      (drafted_logit[c] - row_max[p] >= T ln tau), with p = parent[c], T = params.temperature;
 *   3. per request, from the root repeatedly take the child with the highest drafted logit
 *      (lowest row id on ties) while it is accepted and the promotion budget allows, then
 *      bonus = row_argmax of the last accepted node;
 *   4. draft confidence of each root row and the policy-state update.
 * Workspace: at least asv_workspace_bytes(B, N, H, V) bytes, 256-byte aligned. */
int asv_verify(const asv_verify_args *args, void *workspace, uint64_t workspace_bytes,
               void *stream);

#ifdef __cplusplus
}
#endif

#endif /* ASV_H_ */
