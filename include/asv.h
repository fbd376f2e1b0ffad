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

#define ASV_VERSION 110          /* 1.1.0 */

/* Return codes. */
#define ASV_OK          0
#define ASV_EINVAL     -1        /* bad size, null or misaligned pointer, bad parameter */
#define ASV_EWORKSPACE -2        /* workspace smaller than asv_workspace_bytes() or misaligned */
#define ASV_EHIP       -3        /* a HIP runtime call or kernel launch failed */

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
                                     H > 0 with H % 64 == 0, V > 0 */
  const uint16_t *hidden;         /* [N][H] bf16 final hidden states, 16-byte aligned */
  const uint16_t *w_lm;           /* [V][H] bf16 LM-head weight, 16-byte aligned */
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
  void *k1_begin_event;           /* optional hipEvent_t recorded just before the LM-head
                                     kernel, or NULL */
  void *k1_end_event;             /* optional hipEvent_t recorded just after it, or NULL */
} asv_verify_args;

/* ASV_VERSION of the loaded library. */
int asv_version(void);

/* Static, human-readable text for an ASV_* return code. */
const char *asv_status_string(int code);

/* Details of the most recent ASV_EHIP failure on the calling host thread (the failing launch
 * or runtime call and the HIP error text); "" if none. Valid until the next failing call on
 * this thread. */
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
