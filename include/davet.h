/*
 * davet.h -- C ABI of the DAVET per-denoising-step hot path on MI355X (gfx950).
 *
 * DAVET (Denoising-Aware Visual Evidence Trajectory Allocation) conditions each
 * denoising step of a diffusion vision-language model on one of K evidence views
 * built once from a single visual encoding, chosen per step by an allocation
 * policy.  This library implements, for one GPU:
 *
 *   davet_build_views    the ordered evidence hierarchy (Sec. 4.3)
 *   davet_denoise_step   one pass of the bidirectional denoiser over
 *                        [view | prompt | response] (Sec. 3.1, Eq. 1) with the
 *                        argmax / confidence decoding of masked positions
 *   davet_unmask         confidence-ranked commitment (Eq. 2)
 *   davet_policy_*       the allocation policy (Sec. 4.2, Eqs. 6-9): envelope
 *                        and step on the host, the per-step closed loop also
 *                        on the GPU (davet_policy_step_device)
 *   davet_run_schedule   the whole loop: views once, then T steps
 *
 * Conventions, for every entry point:
 *   - Pointers are DEVICE pointers unless the comment says host.  Arrays are
 *     dense and row-major.  The caller owns every buffer, including the
 *     workspace; the library never frees caller memory and allocates no device
 *     memory (davet_run_schedule uses small host-side vectors; its policy
 *     mode writes into a caller-owned mailbox made once by
 *     davet_mailbox_create).
 *   - Device work is enqueued asynchronously on the given HIP stream.  Only
 *     davet_run_schedule in policy mode synchronises: once per step, on the
 *     GPU kernel that writes the next levels (the next step's launch sizes
 *     depend on them); and davet_fp16_overflow_count, which reads a counter
 *     back to the host.
 *   - Every argument is validated before anything is enqueued; on an error the
 *     call returns a negative davet_status, enqueues nothing, and
 *     davet_last_error() describes the failure (thread-local string).
 *   - Element types: DAVET_F32 = IEEE float32, DAVET_BF16 = bfloat16 bit
 *     patterns, DAVET_F16 = IEEE binary16 bit patterns (both uint16).  The
 *     16-bit modes feed 16-bit operands of that type to the matrix cores with
 *     float32 accumulation; residual streams, softmax statistics and norms
 *     run in float32 in every mode.  A bf16 model is meant to run in the
 *     DAVET_F16 mode: davet_convert rounds its weights to fp16 (a bf16 value
 *     converts exactly when 2^-17 <= |w| <= 65504; smaller ones fall into
 *     fp16's subnormal range and lose bits, |w| <= 2^-25 becomes zero), and
 *     fp16 operands carry 3 more mantissa
 *     bits through the activations at the same matrix-core rate.  The
 *     DAVET_BF16 mode (bf16 activations into the matrix cores) is accurate
 *     to logits rel-RMS <= 1e-2 against a float64 evaluation only for
 *     shallow stacks: measured 6e-3 for one 8B-shaped layer and 2.2e-2 for
 *     32 layers, whose error exceeds that bound; use DAVET_F16 for deep
 *     stacks.
 */
#ifndef DAVET_H
#define DAVET_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum davet_status {
  DAVET_OK = 0,
  DAVET_EINVAL = -1,   /* bad scalar argument or null pointer              */
  DAVET_ESHAPE = -2,   /* unsupported or inconsistent shape                 */
  DAVET_EDTYPE = -3,   /* unsupported element type                          */
  DAVET_ENOMEM = -4,   /* workspace smaller than davet_workspace_bytes()   */
  DAVET_EHIP = -5      /* a HIP runtime call failed                         */
} davet_status;

typedef enum davet_dtype { DAVET_F32 = 0, DAVET_BF16 = 1, DAVET_F16 = 2 } davet_dtype;

/* Limits of this build. */
#define DAVET_MAX_SEQS 64        /* sequences per packed batch            */
#define DAVET_MAX_LEVELS 4       /* K                                     */
#define DAVET_MAX_RESP 1024      /* response length L                     */

/* Evidence realizers (Sec. 4.3: any construction with an ordered
 * evidence-cost hierarchy; pooling is the paper's default, pruning varies
 * the retention ratio, merging the aggregation strength). */
typedef enum davet_realizer {
  DAVET_REALIZER_POOL = 0,   /* per-crop average pooling (and the mixed view) */
  DAVET_REALIZER_PRUNE = 1,  /* nested top-n by token L1 norm                 */
  DAVET_REALIZER_MERGE = 2   /* single-linkage merging by cosine similarity   */
} davet_realizer;
#define DAVET_MAX_REALIZER_GRID 64   /* grid limit of prune and merge */

/* Geometry of one sample's visual encoding v: n_crops crops of grid x grid
 * tokens, each token a d-vector; v is [n_crops*grid*grid, d], crop-major, then
 * row-major inside a crop.  K ordered levels, level K-1 being v itself.
 * mixed_stride: 0 for the pooling pyramid; S >= 2 (K = 3, pooling only) makes
 * level 1 the mixed view of Sec. 4.3 (see davet_build_views).
 * realizer: a davet_realizer; 0 (pooling) when the struct is zero-filled. */
typedef struct davet_view_geom {
  int32_t n_crops;
  int32_t grid;
  int32_t d;
  int32_t K;          /* 1..DAVET_MAX_LEVELS */
  int32_t dtype;      /* davet_dtype of v and of the pooled levels */
  int32_t mixed_stride;
  int32_t realizer;
} davet_view_geom;

/* Denoiser shape.  d = n_heads * head_dim, head_dim in {64, 128} (128 in the
 * 16-bit modes, where d must be a multiple of 128 and ffn of 64); d <= 8192;
 * mask_id in [0, vocab). */
typedef struct davet_model_cfg {
  int32_t n_layers;
  int32_t d;
  int32_t n_heads;
  int32_t head_dim;
  int32_t ffn;
  int32_t vocab;
  int32_t mask_id;
  float rms_eps;
  float rope_theta;
  int32_t dtype;      /* davet_dtype of weights, embeddings and views */
} davet_model_cfg;

/* One layer's parameters (element type = cfg.dtype, out = x W^T):
 *   wqkv [3d, d]  rows: query heads, key heads, value heads (head-major)
 *   wo   [d, d]
 *   wg   [ffn, d] gate, wu [ffn, d] up, wd [d, ffn] down (SwiGLU)
 *   attn_norm, ffn_norm: float32 [d] RMSNorm gains, or NULL for all-ones. */
typedef struct davet_layer_weights {
  const void* wqkv;
  const void* wo;
  const void* wg;
  const void* wu;
  const void* wd;
  const float* attn_norm;
  const float* ffn_norm;
} davet_layer_weights;

/* Layout of the vocabulary-head weights (davet_weights.head_layout).  Both
 * layouts give the same logits and argmaxes bit for bit; the confidences may
 * differ in their last bits (the tiled head sums the exponentials over
 * 256-column vocabulary slabs, the row-major one over 128-column slabs). */
typedef enum davet_head_layout {
  DAVET_HEAD_ROWS = 0,   /* [vocab, d] row-major */
  DAVET_HEAD_TILED = 1   /* 16-bit models only: the output of davet_pack_head */
} davet_head_layout;

/* embed [vocab, d] token embedding; head: untied output head, [vocab, d]
 * row-major or tiled (head_layout); final_norm float32 [d] or NULL; layers:
 * HOST array of n_layers entries. */
typedef struct davet_weights {
  const void* embed;
  const void* head;
  const float* final_norm;
  const davet_layer_weights* layers;
  int32_t head_layout;
} davet_weights;

/* Allocation policy parameters (Sec. 4.2): average budget B, reserve fraction
 * rho, risk strength alpha, operation demand d(o) in [0,1], phase orientation
 * (early != 0: p_t = 1-(t-0.5)/T; else p_t = (t-0.5)/T), K levels. */
typedef struct davet_policy {
  double B;
  double rho;
  double alpha;
  double demand;
  int32_t early;
  int32_t K;
} davet_policy;

const char* davet_last_error(void);
const char* davet_version(void);

/* ---------------------------------------------------------------- views -- */

/* Token counts of the K levels of a geometry (host out[K]).  Level l pools
 * windows of side 2^(K-1-l) per crop with ceil padding:
 * n_l = n_crops * ceil(grid / 2^(K-1-l))^2; the mixed level has
 * n_1 = n_crops * (ceil(grid / 4)^2 + m^2), m = #{o, o+S, ... < grid},
 * o = S / 2.  The prune and merge realizers keep the pooling counts n_l.
 * Errors: EINVAL, ESHAPE (bad K, grid, n_crops, stride or realizer). */
int davet_view_sizes(const davet_view_geom* g, int32_t* n_tokens /*host[K]*/);

/* Lengths of the K member lists of davet_build_views' index maps (host
 * out[K]): n_crops * grid^2 per pyramid or merge level (a partition of the
 * tokens), n_crops * (grid^2 + m^2) for the mixed level, n_l per prune level
 * (one member per kept token). */
int davet_view_map_sizes(const davet_view_geom* g,
                         int32_t* n_members /*host[K]*/);

/* Evidence hierarchy (Sec. 4.3, "Ordered evidence hierarchy"; Sec. 3.2: a full
 * budget leaves v unchanged).  Pooling: level l < K-1 token j is the mean of
 * the in-bounds tokens of its window (divisor = member count), accumulated in
 * float64 and rounded once to the view dtype.  Level K-1 is v itself: nothing
 * is written for it except its (identity) index map.  Prune and merge: the
 * levels given by davet_realizer_maps on davet_realizer_keys, each token the
 * float64 mean of its members in member order, rounded once (a kept token of
 * the prune realizer is copied unchanged).
 *   v            [n_crops*grid*grid, d] (dtype g.dtype), read only
 *   levels       HOST array of K device pointers; levels[l] receives
 *                [n_l, d] for l < K-1; levels[K-1] is ignored (may be NULL)
 *   idx_offsets  HOST array of K device pointers (int32 [n_l + 1]) or NULL;
 *   idx_members  HOST array of K device pointers (int32 [davet_view_map_sizes
 *                entry]) or NULL.  CSR map: token j of level l pools rows
 *                members[offsets[j] .. offsets[j+1]) of v, listed row-major in
 *                the window, ids c*grid*grid + r*grid + s.  Individual entries
 *                may be NULL to skip that level's map.
 * Mixed view (mixed_stride = S >= 2, K = 3; Sec. 4.3: the pooled view
 * augmented with a fixed subset of unpooled tokens): per crop, the level-0
 * tokens (windows of side 4) followed by the raw tokens at rows and columns
 * o, o+S, o+2S, ... (o = S/2), row-major, each a one-member window copied
 * bit for bit from v.
 * scratch: device memory of davet_views_scratch_bytes (NULL / 0 for pooling).
 * Errors: EINVAL (null v / levels entry, misaligned v or level, realizer
 * unknown), ENOMEM (scratch smaller than needed), ESHAPE (grid<1, n_crops<1,
 * K out of range, d % 8 != 0, mixed_stride 1 or < 0, or > 0 with K != 3 or a
 * realizer other than pooling, grid > DAVET_MAX_REALIZER_GRID for prune and
 * merge), EDTYPE. */
int davet_build_views(const davet_view_geom* g, const void* v,
                      void* const* levels, int32_t* const* idx_offsets,
                      int32_t* const* idx_members, void* scratch,
                      size_t scratch_bytes, hipStream_t stream);

/* Device scratch davet_build_views needs for a geometry (0 for pooling): the
 * realizer keys plus the index maps of levels < K-1.  v and the level
 * buffers must be 16-byte aligned; scratch 256-byte aligned.  The scratch is
 * overwritten; nothing is kept in it after the stream reaches the end of
 * the call. */
int davet_views_scratch_bytes(const davet_view_geom* g, size_t* bytes);

/* Number of keys of the prune (n_crops * grid^2, one per token) or merge
 * (n_crops * 2 * grid * (grid - 1), one per grid edge) realizer; 0 for
 * pooling.  Errors: EINVAL, ESHAPE. */
int davet_realizer_key_count(const davet_view_geom* g, int32_t* n_keys);

/* Realizer keys (Sec. 4.3, "Compatible evidence realizers"; the criteria
 * are readings, the paper gives none), float64, device out[n_keys]:
 *   prune  keys[c*grid^2 + i] = sum_j |v[c*grid^2 + i, j]|, the L1 norm of
 *          token i of crop c (exact in any order for fp16 v with d <= 8192);
 *   merge  keys[c*E + e] = cosine similarity of the two tokens of edge e of
 *          crop c, dot / sqrt(|a|^2 |b|^2) (0 if either norm is 0),
 *          E = 2*grid*(grid-1); edges (r,s)-(r,s+1) first at index
 *          r*(grid-1) + s, then (r,s)-(r+1,s) at grid*(grid-1) + r*grid + s.
 * v is [n_crops*grid^2, d] of g.dtype, 16-byte aligned, d % 8 == 0.
 * Errors: EINVAL (null, misaligned, pooling realizer), ESHAPE
 * (grid > DAVET_MAX_REALIZER_GRID), EDTYPE. */
int davet_realizer_keys(const davet_view_geom* g, const void* v,
                        double* keys, hipStream_t stream);

/* For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): davet_build_views with
 * the prune / merge realizers' scratch (davet_views_scratch_bytes: keys and
 * the maps of the pooled levels) in a device array the library holds, of
 * DAVET_STATIC_SCRATCH_BYTES per GPU, kept until the process ends.  Same
 * arguments and results as davet_build_views without scratch; the call
 * allocates nothing.  The first call on a device resolves the array's
 * address there (a one-time set-up step that may load the library's code
 * object: make it before capturing).  All calls on one device share its
 * array: calls that overlap on one device (other streams, other threads)
 * race; consecutive calls on one stream are safe (everything a call reads
 * from the array it first writes).  Pooling needs no scratch and never
 * touches the array.  Errors: as davet_build_views, and ENOMEM when the
 * geometry needs more scratch than the maximum (e.g. the merge realizer on
 * more than ~40 crops of a 64 x 64 grid). */
#define DAVET_STATIC_SCRATCH_BYTES (4u << 20)
int davet_build_views_static(const davet_view_geom* g, const void* v,
                             void* const* levels, int32_t* const* idx_offsets,
                             int32_t* const* idx_members, hipStream_t stream);

/* Index maps of all K levels from given keys (device float64 [n_keys]),
 * deterministic for identical keys.  Keys are ordered larger first, equal
 * keys by lower index, NaN as -inf, -0 as +0.  Per crop and level l with
 * n = ceil(grid / 2^(K-1-l))^2 tokens (the pooling counts):
 *   prune  the n tokens first in key order, listed by index, one member
 *          each (nested over levels);
 *   merge  edges are taken in key order and each edge joining two groups
 *          merges them until n groups remain, for l = K-2 down to 0
 *          (single linkage; coarser groups are unions of finer ones);
 *          groups listed by smallest member, members ascending.
 * Level K-1 gets the identity map.  idx_offsets[l] ([n_l + 1]) and
 * idx_members[l] (davet_view_map_sizes entry) are device pointers in HOST
 * arrays of K; a NULL entry skips that level.  Errors as
 * davet_realizer_keys. */
int davet_realizer_maps(const davet_view_geom* g, const double* keys,
                        int32_t* const* idx_offsets,
                        int32_t* const* idx_members, hipStream_t stream);

/* Element-type conversion of n values, rounding to nearest even (e.g. a bf16
 * checkpoint into the fp16 operand mode: a bf16 value converts exactly when
 * 2^-17 <= |x| <= 65504, smaller ones lose bits in fp16's subnormal range).  src and dst are device buffers of n elements of their
 * dtypes and must not overlap.  Errors: EINVAL (null, overlap), EDTYPE. */
int davet_convert(const void* src, int32_t src_dtype, void* dst,
                  int32_t dst_dtype, size_t n, hipStream_t stream);

/* Tiled copy of a 16-bit vocabulary head for the head kernel (a one-time
 * model-load transform; the logits are bit-identical to those of the
 * row-major head).  The tiled head is a sequence of 128 x 64 tiles, k-chunk
 * major, so that every vocabulary slab reads chunk c of its rows from one
 * contiguous region while all slabs stream chunk c at the same time:
 *   tiled[((c * S + s) * 128 + r) * 64 + j] = head[(128 s + r) * d + 64 c + j]
 * with S = ceil(vocab / 128) slabs, c < d / 64, r < 128, j < 64; rows past
 * vocab are zero.  src [vocab, d] and dst [davet_head_tiled_elems(vocab, d)]
 * are device buffers of dtype (DAVET_BF16 or DAVET_F16) and must not overlap.
 * Errors: EINVAL (null, overlap), ESHAPE (vocab < 1, d < 64, d % 64 != 0),
 * EDTYPE. */
size_t davet_head_tiled_elems(int32_t vocab, int32_t d);
int davet_pack_head(const void* src, void* dst, int32_t vocab, int32_t d,
                    int32_t dtype, hipStream_t stream);

/* ------------------------------------------------------------- denoiser -- */

/* Workspace bytes davet_denoise_step needs for at most max_tokens packed
 * tokens (sum over sequences of n_view + prompt + L), max_seqs sequences and
 * response length L.  The workspace must be 256-byte aligned. */
int davet_workspace_bytes(const davet_model_cfg* cfg, int32_t max_tokens,
                          int32_t max_seqs, int32_t L, size_t* bytes /*host*/);

/* One denoising step for a packed batch of n_seqs independent sequences
 * (Sec. 3.1, Eq. 1, with the view v_t of Sec. 3.2).  Sequence s is
 *   [ view_ptrs[s] (n_view[s] rows) | E[prompt ids cu_prompt[s]..cu_prompt[s+1]) |
 *     E[resp_ids[s*L + i]], or E[mask_id] where resp_masked[s*L + i] != 0 ]
 * at rotary positions 0..N_s-1, run through cfg.n_layers pre-norm layers with
 * NON-causal attention inside each sequence only (Sec. 1: bidirectional).
 * For every masked response position the final-normed hidden state is projected
 * on the vocabulary and decoded at temperature 0 (Sec. 5.1):
 *   argmax_out[s*L+i] = argmax over w != mask_id (lowest id on ties)
 *   conf_out[s*L+i]   = max softmax probability, [MASK] excluded from the
 *                       normaliser: 1 / sum_{w != mask} exp(l_w - l_argmax)
 * Committed (unmasked) positions get conf = -inf and argmax = -1.
 *   view_ptrs, n_view, cu_prompt: HOST arrays; view rows have dtype cfg.dtype.
 *   prompt_ids int32 [cu_prompt[n_seqs]]; resp_ids int32 [n_seqs*L];
 *   resp_masked uint8 [n_seqs*L]; conf_out float [n_seqs*L];
 *   argmax_out int32 [n_seqs*L];
 *   logits_out float [n_seqs*L, vocab] or NULL: when given, the logits of
 *   masked positions are stored in their rows (other rows untouched).
 *   Weight matrices, norm vectors and view rows are read with 16-byte
 *   vector loads: their pointers must be 16-byte aligned (EINVAL otherwise).
 * Errors: EINVAL, ESHAPE (head_dim, d, ffn, n_seqs, L or token counts out of
 * range), EDTYPE, ENOMEM (ws_bytes too small or workspace misaligned). */
int davet_denoise_step(const davet_model_cfg* cfg, const davet_weights* w,
                       int32_t n_seqs, const void* const* view_ptrs,
                       const int32_t* n_view, const int32_t* prompt_ids,
                       const int32_t* cu_prompt, const int32_t* resp_ids,
                       const uint8_t* resp_masked, int32_t L, float* conf_out,
                       int32_t* argmax_out, float* logits_out, void* workspace,
                       size_t ws_bytes, hipStream_t stream);

/* Number of non-finite values the 16-bit modes stored as GEMM outputs in the
 * last davet_denoise_step on this workspace, or over all the steps of the
 * last davet_run_schedule on it.  The counted stores are the projections'
 * 16-bit outputs: Q/K/V (after rotary embedding) and the SwiGLU product fed
 * to the down projection.  In DAVET_F16 a value beyond +-65504 becomes +-inf
 * there, so a nonzero count means the fp16 range was too small for this model
 * and input (run it in DAVET_F32, or DAVET_BF16 for a shallow stack).  The
 * other 16-bit tensors are bounded by these or by a norm: attention outputs
 * are convex combinations of V rows, and normed rows are at most
 * sqrt(d) * max|gain| in magnitude.  The residual stream and the logits are
 * float32 and not counted; a DAVET_F32 model always reads 0.
 *   workspace: the same 256-byte aligned workspace the step ran on (the
 *   counter is its first 4 bytes); count: HOST int32.
 * Enqueues a 4-byte read on `stream` and waits for it.  Errors: EINVAL (null
 * or misaligned pointer), EHIP (the copy or the wait failed). */
int davet_fp16_overflow_count(const void* workspace, int32_t* count /*host*/,
                              hipStream_t stream);

/* Key-range split of the 16-bit attention (process-wide setting).  A query
 * tile's workgroup normally sweeps every key of its sequence (Sec. 3.1:
 * bidirectional attention, every query sees every key).  When the ragged
 * last query tiles of a launch would run as a thin extra round behind the
 * full tiles, the library divides their keys among up to 8 workgroups, each
 * writing fp32 partial softmax statistics and outputs into the workspace,
 * and a merge kernel combines the pieces in a fixed order, so the result does
 * not depend on timing; only the summation order differs from the unsplit
 * launch.
 *   mode 0: automatic (default); 1: never split; 2..8: split every query
 *   tile into `mode` key ranges (a testing and tuning override; launches
 *   whose partials would not fit in the workspace stay unsplit).
 * Errors: EINVAL (mode outside [0, 8]). */
int davet_set_attention_split(int32_t mode);

/* --------------------------------------------------------------- unmask -- */

/* Confidence-ranked commitment, Eq. (2) (Sec. 5.1: confidence ranking).  Per
 * sequence s, among positions with resp_masked != 0, the k_s = min(k, |M|)
 * positions ranked first by (conf descending, position ascending) -- NaN ranks
 * with -inf, below every number -- are committed: resp_ids[i] = argmax[i],
 * resp_masked[i] = 0.  Other positions are untouched.
 *   conf float [n_seqs*L], argmax int32 [n_seqs*L] (read only)
 *   resp_ids int32 [n_seqs*L], resp_masked uint8 [n_seqs*L] (updated in place)
 *   selected int32 [n_seqs*k] or NULL: committed positions of each sequence in
 *   rank order, padded with -1.
 * Errors: EINVAL (k < 1, null pointers), ESHAPE (L out of range, n_seqs < 1). */
int davet_unmask(int32_t n_seqs, int32_t L, int32_t k, const float* conf,
                 const int32_t* argmax, int32_t* resp_ids, uint8_t* resp_masked,
                 int32_t* selected, hipStream_t stream);

/* ------------------------------------------------------ policy (host) -- */

/* Demand prior d(o) of Appendix A, Table A: category 0 lexical readout 1.000,
 * 1 numerical reasoning 0.941, 2 entity grounding 0.824, 3 binary decision
 * 0.647, 4 general understanding 0.529.  Returns a negative value for an
 * unknown category. */
double davet_demand_prior(int32_t category);

/* Operation parser g (App. A, "Operation Parser and Demand Prior"): the
 * category of a query text (NUL-terminated, any case), host only.  The
 * query is lowercased, generic conversation wrappers ("<image>", "answer
 * the question using a single word or phrase", "in the image", ...) are
 * dropped and the words are matched against the cue families in the
 * appendix's order -- binary decision (auxiliary- or modal-initial), numerical
 * reasoning, lexical readout, entity grounding -- the first match deciding;
 * otherwise general understanding.  The cue phrase lists are this library's
 * reading (the appendix describes the families, not the lists).  *category
 * uses the indices of davet_demand_prior.  Errors: EINVAL (null). */
int davet_parse_operation(const char* query, int32_t* category /*host*/);

/* Evidence envelope, Eq. (6): lower = N(p; (1-rho)B), upper = N(p;
 * [1-rho+rho d]B), with p the phase profile of Sec. 4.2 and N the rescale-and-
 * clip normaliser (exact scale: min(1, s p_t), mean = beta; beta >= 1 gives
 * ones, beta <= 0 zeros).  Double precision, evaluated without contraction.
 * lower, upper: HOST double [T].  Errors: EINVAL (T < 1, null, non-finite). */
int davet_policy_envelope(const davet_policy* pol, int32_t T,
                          double* lower, double* upper);

/* Budget and level of step t (1-based): r_t by Eq. (7) (r_1 = 1), b_t by
 * Eq. (8), level by Eq. (9) generalised to K levels (count of thresholds j/K,
 * j = 1..K-1, that are <= b_t).  lower/upper from davet_policy_envelope.
 * b_t, level, r_t: HOST outputs (r_t may be NULL). */
int davet_policy_step(const davet_policy* pol, int32_t t, int32_t T,
                      const double* lower, const double* upper,
                      double cbar_prev, double churn_prev, double* b_t,
                      int32_t* level, double* r_t);

/* Generation-state signals after a step (Sec. 4.2, before Eq. 7), all HOST
 * arrays of L entries.  cbar = mean of conf over positions still masked after
 * the step's commitment (masked_after != 0), summed in ascending position
 * order; churn = fraction of those positions whose argmax differs from
 * argmax_prev (0 on the first step: argmax_prev == NULL).  Empty set: 0, 0. */
int davet_step_stats(int32_t L, const float* conf, const int32_t* argmax,
                     const int32_t* argmax_prev, const uint8_t* masked_after,
                     double* cbar, double* churn);

/* The closed loop on the GPU (Sec. 4.2): davet_step_stats of every sample
 * after step t's commitment followed by davet_policy_step for step t+1, with
 * bit-identical results (the same float64 operations in the same order).
 *   n_seqs samples of L response positions; 1 <= t < T.
 *   pols, lower, upper: HOST (lower/upper [n_seqs * T] from
 *     davet_policy_envelope, sample s at s*T); every pols[s].K equal.
 *   conf, argmax (step t), argmax_prev (step t-1; NULL exactly when t = 1),
 *   masked_after: DEVICE [n_seqs * L], sample-major.
 *   level_out, budget_out (and r_out unless NULL): DEVICE or pinned host
 *     [n_seqs], the level, b_{t+1} and r_{t+1} of each sample.
 * Errors: EINVAL (null, t out of range, argmax_prev inconsistent with t, K
 * differs or out of range), ESHAPE (n_seqs, L). */
int davet_policy_step_device(int32_t n_seqs, int32_t L, int32_t t, int32_t T,
                             const davet_policy* pols, const double* lower,
                             const double* upper, const float* conf,
                             const int32_t* argmax, const int32_t* argmax_prev,
                             const uint8_t* masked_after, int32_t* level_out,
                             double* budget_out, double* r_out,
                             hipStream_t stream);

/* ------------------------------------------------------------- schedule -- */

/* Mailbox of the policy-mode loop (Sec. 4.2's closed loop): after every
 * step the GPU writes the next levels and budgets of each sample into it,
 * then a stamp the host waits for.  davet_mailbox_create is a one-time
 * set-up call: it allocates a few hundred bytes of pinned, host-coherent
 * memory (hipHostMalloc) that the caller owns until davet_mailbox_destroy,
 * which first synchronises the device (a policy step still queued may write
 * the mailbox) and then frees it.  A mailbox serves one davet_run_schedule
 * call at a time (calls that overlap on one mailbox race); each call uses
 * stamps no earlier call on that mailbox used.  Host only.
 * Errors: EINVAL (null out), ENOMEM, EHIP. */
typedef struct davet_mailbox davet_mailbox;
int davet_mailbox_create(davet_mailbox** out /*host*/);
int davet_mailbox_destroy(davet_mailbox* mailbox);   /* NULL: no-op */

/* Host-side limit (seconds, default 120) on each wait of davet_run_schedule
 * for a step's published levels; a longer wait returns DAVET_EHIP while the
 * stream may still be running (synchronise it before reusing the mailbox,
 * the workspace or the outputs).  Process-wide.  Errors: EINVAL (not
 * positive and finite). */
int davet_set_wait_limit(double seconds);

/* The whole DAVET loop for a packed batch (Sec. 3.1 and Sec. 4; Fig. 2):
 * davet_build_views once per sequence into view_bufs, then for t = 1..T:
 * choose each sequence's level -- fixed_levels[s*T + t-1] when fixed_levels is
 * given, else the policy pols[s] (Eqs. 7-9) from the signals of step t-1 --
 * davet_denoise_step, davet_unmask with k.  In policy mode each step but the
 * last ends with the device policy step (as davet_policy_step_device,
 * writing the next levels and budgets into the mailbox) and a host wait for
 * its stamp, bounded by davet_set_wait_limit; the levels and budgets equal
 * those of davet_step_stats + davet_policy_step on the same signals bit for
 * bit.  The call allocates and frees no host or device memory.
 *   geoms: HOST [n_seqs] (d and dtype must match cfg)
 *   visual: HOST [n_seqs] device pointers to each v
 *   view_bufs: HOST [n_seqs*(K-1)] device pointers, pooled level l of
 *              sequence s at view_bufs[s*(K-1) + l], sized by davet_view_sizes
 *   prompt_ids/cu_prompt as in davet_denoise_step (cu_prompt on the HOST)
 *   resp_ids / resp_masked: device, [n_seqs*L], in/out (normally all-masked
 *              on entry)
 *   pols: HOST [n_seqs] or NULL; fixed_levels: HOST [n_seqs*T] or NULL; exactly
 *         one of the two must be given.
 *   levels_out int32 / budgets_out double: HOST [n_seqs*T] or NULL
 *         (budgets are NaN in fixed mode)
 *   conf_trace float / argmax_trace int32: device [T, n_seqs*L] or NULL.
 *   mailbox: from davet_mailbox_create; required in policy mode with T > 1,
 *            ignored (may be NULL) otherwise.
 * Errors: as the calls it makes; EINVAL for a bad schedule argument or a
 * missing mailbox; EHIP when a wait for published levels fails or exceeds
 * the wait limit. */
int davet_run_schedule(const davet_model_cfg* cfg, const davet_weights* w,
                       int32_t n_seqs, const davet_view_geom* geoms,
                       const void* const* visual, void* const* view_bufs,
                       const int32_t* prompt_ids, const int32_t* cu_prompt,
                       int32_t L, int32_t T, int32_t k,
                       const davet_policy* pols, const int32_t* fixed_levels,
                       int32_t* resp_ids, uint8_t* resp_masked,
                       int32_t* levels_out, double* budgets_out,
                       float* conf_trace, int32_t* argmax_trace,
                       davet_mailbox* mailbox, void* workspace,
                       size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------ profiling -- */

/* Per-kernel-class timing with HIP events recorded around every launch on the
 * launch stream (for the measurement harness).  davet_prof_enable(n) reserves
 * event pairs for n launches (host-side and HIP event objects, created here,
 * not in the steady state) and starts recording; davet_prof_enable(0) stops
 * and releases them.  davet_prof_read synchronises on the recorded events and
 * fills, per kernel class c < n_classes, the launch count and summed
 * milliseconds; names via davet_prof_class_name.  Returns the number of
 * classes, or a negative status.  davet_prof_only(c) restricts recording to
 * launches of class c (so that a timed run carries events around one kernel
 * class only); -1 records every class again. */
int davet_prof_enable(int32_t max_launches);
int davet_prof_reset(void);
int davet_prof_only(int32_t cls);
int davet_prof_read(int32_t n_classes, int64_t* counts /*host*/,
                    double* total_ms /*host*/);
const char* davet_prof_class_name(int32_t cls);

#ifdef __cplusplus
}
#endif
#endif /* DAVET_H */
