/*
 * dv.h — C ABI of the Deja Vu decode hot path for AMD Instinct MI355X (gfx950).
 *
 * Deja Vu (Liu et al., ICML 2023, arXiv 2310.17157) skips, for each generated
 * token, the attention heads and MLP neurons that a cheap predictor deems
 * irrelevant to that token ("contextual sparsity"). This library implements the
 * decode-time hot path on one GPU:
 *   - the low-rank sparsity predictors (two thin GEMVs, then top-k or threshold
 *     selection): dv_predict_mlp, dv_predict_heads;
 *   - the sparsified MLP of Eq. (1): dv_sparse_mlp (fp16/fp32 weights, one token
 *     or a batch of up to 32), dv_sparse_mlp_q4 (4-bit weights, Section 5.2);
 *   - the sparsified multi-head attention of Eq. (2) over a KV cache:
 *     dv_sparse_attn, and dv_sparse_attn_kvfill with the missing-KV rule of
 *     Section 4.2;
 *   - one whole decoder layer with predictors, layer norms and residuals
 *     (Section 4.3): dv_sparse_block, and dv_sparse_block_noalloc for callers
 *     that cannot allocate a workspace;
 *   - several layers of one token with the cross-layer look-ahead of Section 4.3:
 *     dv_sparse_decode.
 * Aids: dv_set_launch_events / dv_launch_label (per-launch timing) and
 * dv_stream_read (a plain streaming read, the measured bandwidth ceiling).
 *
 * Conventions shared by every entry point
 *   Memory.   Every array pointer is a DEVICE pointer owned by the caller, except
 *             dv_kv.pos, which is a HOST array (the attention grid is sized from
 *             it on the host). The library never allocates or frees memory on
 *             these paths and keeps no per-call state; scratch space is the
 *             caller's workspace `ws` of at least the size returned by the
 *             matching *_workspace_bytes query (256-byte aligned). Calls that
 *             share a workspace must be ordered on one stream. Global state is
 *             limited to a thread-safe per-device cache (CU count, LDS size,
 *             which kernels had their LDS limit raised) and the per-thread
 *             launch-event hook below; entry points may be called from several
 *             threads and on several devices.
 *   Layout.   Row-major. A weight row is 16-byte aligned: base pointers must be
 *             16-byte aligned and d (and r for predictors) a multiple of 8 for
 *             fp16 or 4 for fp32 elements.
 *   Types.    Weights and predictor factors are fp16 or fp32 (dv_dtype); biases,
 *             layer-norm parameters, hidden states and outputs are fp32; index
 *             sets are int32. Arithmetic accumulates in fp32.
 *   Streams.  `stream` is a hipStream_t (NULL = the null stream). Each call
 *             validates its arguments on the host, synchronously, before any
 *             device work; on success it enqueues its kernels and returns DV_OK
 *             without waiting. Results are valid in stream order.
 *   Errors.   A failed check returns its dv_status and enqueues nothing. A failed
 *             launch returns DV_ERR_HIP. No C++ exception crosses the ABI.
 *   Sets.     An index set is int32, strictly ascending, within [0, n). Selection
 *             outputs always satisfy this. Consumers trust their input sets; an
 *             out-of-range index is clamped into range (no fault, unspecified
 *             result) unless DV_VALIDATE is set, in which case the set is checked
 *             on the device first, the call waits for that check, and a bad set
 *             returns DV_ERR_INDEX with no compute enqueued.
 *   Outputs.  Overwritten, never accumulated. Inputs and outputs must not alias.
 *   Numerics. All reductions run in a fixed order: two identical calls produce
 *             bitwise identical outputs (DV_DETERMINISTIC is always honoured).
 */
#ifndef DV_H
#define DV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DV_ABI_VERSION 1

typedef enum dv_status {
  DV_OK = 0,
  DV_ERR_NULL = 1,        /* a required pointer is NULL */
  DV_ERR_SHAPE = 2,       /* inconsistent or out-of-range sizes (k > n, pos >= cap, ...) */
  DV_ERR_DTYPE = 3,       /* unknown dv_dtype */
  DV_ERR_ALIGN = 4,       /* a pointer or row is not 16-byte aligned */
  DV_ERR_WORKSPACE = 5,   /* workspace NULL, too small or not 256-byte aligned */
  DV_ERR_INDEX = 6,       /* DV_VALIDATE only: an index set is not ascending within [0, n) */
  DV_ERR_HIP = 7,         /* a HIP runtime call or kernel launch failed */
  DV_ERR_UNSUPPORTED = 8, /* a valid request outside what this build implements */
  DV_ERR_ARG = 9          /* an invalid mode or flag value */
} dv_status;

/* DV_Q4: 4-bit weights (W4A16) in the dv_mlp_q4 layout, for dv_sparse_mlp_q4 only. */
typedef enum dv_dtype { DV_F32 = 0, DV_F16 = 1, DV_Q4 = 2 } dv_dtype;
/* sigma of Eq. (1) (Section 2.3 names ReLU and GeLU): dv_mlp.act, dv_mlp_q4.act. */
enum { DV_ACT_RELU = 0, DV_ACT_GELU = 1 };

/* Selection rule (Section 4.1; Algorithm 1 labels s >= t as positive). */
enum { DV_SELECT_TOPK = 0, DV_SELECT_THRESHOLD = 1 };
/* Which hidden state feeds the neuron predictor in dv_sparse_block (Section 4.3):
 * LOOKAHEAD = LN1(y), the attention block's input, so the prediction can run ahead
 * of the attention; SEQUENTIAL = LN2(y~), the MLP block's own input. */
enum { DV_LOOKAHEAD = 0, DV_SEQUENTIAL = 1 };
/* Batch > 1 (Section 5.2, Appendix C.1): UNION runs every sequence on the union of
 * the batch's neuron sets (one skinny GEMM over the union's rows); MASKED gives each
 * sequence only its own neurons. */
enum { DV_MLP_UNION = 0, DV_MLP_MASKED = 1 };
/* Flags. */
enum { DV_DETERMINISTIC = 1u << 0, DV_VALIDATE = 1u << 1 };

/* Two-layer low-rank sparsity predictor (Section 4.1 "Design", Section 4.2
 * "Approach"): scores s = (x A) B, A = AT^T (d x r), B = BT^T (r x n_out); no hidden
 * activation and no bias. n_out is the neuron count N (MLP) or the head count H. */
typedef struct dv_predictor {
  int32_t d;          /* input width */
  int32_t r;          /* rank (hidden width of the predictor) */
  int32_t n_out;      /* number of scored items */
  int32_t wtype;      /* dv_dtype of AT and BT */
  const void *AT;     /* [r][d]; row m = column m of A */
  const void *BT;     /* [n_out][r]; row i = column i of B */
} dv_predictor;

/* ReLU MLP of Eq. (1) with its weights stored transposed (Section 4.4 "Memory
 * coalescing"): neuron i's input weights W^1_i and output weights W^2_i are each one
 * contiguous row. */
typedef struct dv_mlp {
  int32_t d;          /* model width */
  int32_t n;          /* neurons N */
  int32_t wtype;      /* dv_dtype of W1T and W2T */
  int32_t act;        /* DV_ACT_RELU (0, OPT) or DV_ACT_GELU (exact, x * Phi(x)) */
  const void *W1T;    /* [n][d]; row i = W^1_i */
  const float *b1;    /* [n] or NULL */
  const void *W2T;    /* [n][d]; row i = W^2_i */
  const float *b2;    /* [d] or NULL; added once */
} dv_mlp;

/* Multi-head attention of Eq. (2): per head i, W^Q_i, W^K_i, W^V_i (d x dh) stored as
 * the row block [i*dh, (i+1)*dh) of Wq/Wk/Wv (the nn.Linear layout), and W^O_i
 * (dh x d) as the same row block of WoT. */
typedef struct dv_attn {
  int32_t d;          /* model width */
  int32_t H;          /* heads */
  int32_t dh;         /* head width */
  int32_t wtype;      /* dv_dtype of Wq, Wk, Wv, WoT */
  const void *Wq, *Wk, *Wv;        /* [H*dh][d] */
  const float *bq, *bk, *bv;       /* [H*dh] or NULL */
  const void *WoT;                 /* [H*dh][d] */
  const float *bo;                 /* [d] or NULL; added once */
} dv_attn;

/* KV cache: the keys X W^K_i and values X W^V_i of the attended tokens, per head. */
typedef struct dv_kv {
  int32_t B;          /* sequences */
  int32_t H;          /* heads (= dv_attn.H) */
  int32_t dh;         /* head width (= dv_attn.dh) */
  int32_t cap;        /* rows per (sequence, head) */
  int32_t ktype;      /* dv_dtype of K and V */
  int32_t reserved;   /* must be 0 */
  void *K, *V;        /* [B][H][cap][dh], device */
  const int32_t *pos; /* HOST [B]: row of the current token; attention covers rows 0..pos */
} dv_kv;

/* Pre-layer-norm parameters (biased variance). g1 == NULL means no normalisation
 * before the attention block; g2 == NULL none before the MLP. be* may be NULL (0). */
typedef struct dv_ln {
  const float *g1, *be1, *g2, *be2;   /* [d] each */
  float eps;
} dv_ln;

const char *dv_status_string(int32_t status);
int32_t dv_abi_version(void);

/* Per-launch timing (tracing aid). While armed on the calling thread, every entry point
 * called on that thread times its launches (for the i-th timed launch, i < n_pairs):
 * events[2*i] takes the start time of the launch's first kernel and events[2*i+1] the
 * end time of its last kernel, both stamped by those kernels' own dispatches
 * (hipExtLaunchKernel) on the entry point's stream; a launch that runs no kernel
 * records the two events back to back. Events are hipEvent_t handles created by the
 * caller. A launch is timed if `only` is NULL or equals its label. The number of
 * launches of the latest call is stored in *n_launched; dv_launch_label(i) names its
 * i-th launch. Pass events == NULL to disarm. Returns DV_ERR_SHAPE if n_pairs < 0. */
dv_status dv_set_launch_events(void **events, int32_t n_pairs, int32_t *n_launched, const char *only);
const char *dv_launch_label(int32_t i);

/* Measured ceiling (measurement aid, not part of the method): reads `bytes` bytes of
 * the device buffer `buf` once, contiguously, with the same 16-byte non-temporal loads
 * the gathered kernels use, and nothing else. `bytes` must be a multiple of 16 and
 * `buf` 16-byte aligned (else DV_ERR_ALIGN); `sink` is one device float that is never
 * written in practice (it keeps the loads from being removed). The gathered kernels'
 * bandwidth is reported against this plain stream of the same byte count. */
dv_status dv_stream_read(const void *buf, size_t bytes, float *sink, void *stream);

/* ---------------------------------------------------------------- predictors
 * dv_predict_mlp / dv_predict_heads: S = select(s), s = (x A) B (Sections 4.1-4.2).
 *   x      [B][d] fp32 device: the predictor input (already normalised, if any).
 *   mode   DV_SELECT_TOPK: the k highest scores, ties to the lower index, for
 *          0 <= k <= n_out (else DV_ERR_SHAPE; k = n_out gives 0..n_out-1);
 *          DV_SELECT_THRESHOLD: every i with s_i >= thresh (k ignored). Scores are
 *          ordered as floats with -0 = +0; a NaN score gives an unspecified set.
 *   idx    [B][cap_idx] int32 device, out: each sequence's set, ascending. Top-k
 *          needs cap_idx >= k. Threshold mode writes the first cap_idx members.
 *   count  [B] int32 device, out (may be NULL for top-k): |S| (threshold mode: the
 *          full count, which may exceed cap_idx).
 *   scores [B][n_out] fp32 device, out, or NULL: the raw scores s.
 * Limits: n_out <= 2^26 for selection. Both functions compute the same thing;
 * they differ only in launch tuning for a large (neurons) or small (heads) n_out.
 */
size_t dv_predict_workspace_bytes(const dv_predictor *p, int32_t B);
dv_status dv_predict_mlp(const dv_predictor *p, const float *x, int32_t B, int32_t mode,
                         int32_t k, float thresh, int32_t *idx, int32_t cap_idx, int32_t *count,
                         float *scores, void *ws, size_t ws_bytes, uint32_t flags, void *stream);
dv_status dv_predict_heads(const dv_predictor *p, const float *x, int32_t B, int32_t mode,
                           int32_t k, float thresh, int32_t *idx, int32_t cap_idx, int32_t *count,
                           float *scores, void *ws, size_t ws_bytes, uint32_t flags, void *stream);

/* --------------------------------------------------------------- sparse MLP
 * dv_sparse_mlp: out[b] = MLP_S(x[b]) = b2 + sum_{i in S} sigma(x[b] . W^1_i + b1_i) W^2_i
 * (Eq. (1); sigma = ReLU or GeLU by m->act), without any residual.
 *   idx          device int32: idx_per_seq == 0: one set idx[n_idx] shared by all B
 *                sequences; idx_per_seq == 1: idx[B][n_idx], one set per sequence.
 *   batch_mode   with per-sequence sets and B > 1: DV_MLP_UNION or DV_MLP_MASKED.
 * Each selected row of W1T and W2T is read from HBM once per call, whatever B is.
 * Limits: B > 1 needs B <= 32, fp16 weights and n <= 131072 (else DV_ERR_UNSUPPORTED).
 */
size_t dv_sparse_mlp_workspace_bytes(const dv_mlp *m, int32_t B, int32_t n_idx, int32_t idx_per_seq);
dv_status dv_sparse_mlp(const dv_mlp *m, const float *x, int32_t B, const int32_t *idx,
                        int32_t n_idx, int32_t idx_per_seq, int32_t batch_mode, float *out,
                        void *ws, size_t ws_bytes, uint32_t flags, void *stream);

/* ------------------------------------------------------ 4-bit sparse MLP (W4A16)
 * dv_sparse_mlp_q4: dv_sparse_mlp for one token (B = 1) with 4-bit weights, the W4A16
 * setting of Section 5.2 ("Compatibility with Quantization"): out = b2 + sum_{i in S}
 * sigma(x . W^1_i + b1_i) W^2_i, where element j of a stored row is s_{j/32} (q_j - 8):
 * 4-bit codes q_j, two per byte (even element in the low nibble), and one fp16 scale per
 * block of 32 elements. Each selected row is 0.5625 d bytes (d / 2 of codes, d / 16 of
 * scales) instead of 2 d in fp16. Arithmetic in fp32.
 *   W1T, W2T  [n][d/2] uint8 device, 16-byte aligned rows (d a multiple of 32).
 *   S1, S2    [n][d/32] fp16 device: row i's block scales.
 *   act       DV_ACT_RELU or DV_ACT_GELU.
 * idx, n_idx, out, ws, flags as for dv_sparse_mlp with B = 1. */
typedef struct dv_mlp_q4 {
  int32_t d, n;       /* model width (multiple of 32), neurons */
  int32_t act;        /* DV_ACT_RELU or DV_ACT_GELU */
  int32_t reserved;   /* must be 0 */
  const void *W1T, *S1;
  const float *b1;    /* [n] or NULL */
  const void *W2T, *S2;
  const float *b2;    /* [d] or NULL */
} dv_mlp_q4;
size_t dv_sparse_mlp_q4_workspace_bytes(const dv_mlp_q4 *m, int32_t n_idx);
dv_status dv_sparse_mlp_q4(const dv_mlp_q4 *m, const float *x, const int32_t *idx, int32_t n_idx, float *out,
                           void *ws, size_t ws_bytes, uint32_t flags, void *stream);

/* ---------------------------------------------------------- sparse attention
 * dv_sparse_attn: out[b] = bo + sum_{i in S_A^b} H_i(x[b]) W^O_i (Eq. (2) with a
 * `scale` on the logits; scale = 1 is Eq. (2) literally, 1/sqrt(dh) is the usual
 * convention), without any residual.
 *   heads   [B][n_heads] int32 device: each sequence's head set S_A^b.
 *   kv      the cache; for every b and every i in S_A^b the fresh key and value of
 *           x[b] are written at row pos[b] (Section 4.2: keys and values only for
 *           the selected heads; other heads' rows are left untouched), then head i
 *           attends over rows 0..pos[b].
 */
size_t dv_sparse_attn_workspace_bytes(const dv_attn *a, const dv_kv *kv, int32_t B, int32_t n_heads);
dv_status dv_sparse_attn(const dv_attn *a, const float *x, int32_t B, const dv_kv *kv,
                         const int32_t *heads, int32_t n_heads, float scale, float *out,
                         void *ws, size_t ws_bytes, uint32_t flags, void *stream);

/* ------------------------------------------ sparse attention, missing keys and values
 * dv_sparse_attn_kvfill: dv_sparse_attn for one sequence (kv->B = 1) with the missing-KV
 * rule of Section 4.2 ("Approach"). Only selected heads write their key and value of a
 * token, so a head selected now may lack rows of past tokens; the attention input of
 * every token is kept, and the missing rows of the selected heads are computed from it
 * (K[h][t] = Y[t] W^K_h + bk_h, likewise V) before those heads attend.
 *   x      [d] fp32 device: this token's attention input (normalised, as for dv_sparse_attn).
 *   Y      [cap][d] device, in/out, in the cache's type (kv->ktype: fp16 or fp32, like
 *          the keys and values computed from it): the kept inputs; the call writes
 *          Y[pos] = x, rounded to nearest even for fp16. 16-byte aligned.
 *   valid  [H][cap] uint8 device, in/out: 1 where row t of head h holds token t's key
 *          and value. On return valid[h][0..pos] = 1 for every selected head and
 *          valid[h][pos] = 0 for the others; rows above pos are not touched. A sequence
 *          starts with 1 for the rows its prompt filled and 0 elsewhere.
 *   out, heads, n_heads, scale, ws, flags as for dv_sparse_attn (workspace: the
 *          dv_sparse_attn_workspace_bytes query with B = 1).
 * Cost: one launch more than dv_sparse_attn; it reads no weights when no selected head
 * misses a row, otherwise each selected head's W^K and W^V rows once per 4 missing
 * positions. Limits: pos <= 32768 (else DV_ERR_UNSUPPORTED). */
dv_status dv_sparse_attn_kvfill(const dv_attn *a, const float *x, const dv_kv *kv, void *Y, uint8_t *valid,
                                const int32_t *heads, int32_t n_heads, float scale, float *out, void *ws,
                                size_t ws_bytes, uint32_t flags, void *stream);

/* ------------------------------------------------------------- decoder layer
 * dv_sparse_block: one decoder layer for one token per sequence (Section 4.3):
 *   S_A  = top-k_heads(SP_A(LN1(y)))
 *   y~   = y + MHA_{S_A}(LN1(y))
 *   S_M  = top-k_mlp(SP_M(LN1(y)))   (mode DV_LOOKAHEAD)
 *        = top-k_mlp(SP_M(LN2(y~)))  (mode DV_SEQUENTIAL)
 *   y^   = y~ + MLP_{S_M}(LN2(y~))   -> x_out
 *   pa, pm      head and neuron predictors (pa->n_out = H, pm->n_out = N).
 *   heads_out   [B][k_heads] or NULL: S_A per sequence, ascending.
 *   idx_out     [B][k_mlp] or NULL: S_M per sequence, ascending.
 *   batch_mode  B > 1: DV_MLP_UNION or DV_MLP_MASKED (see above).
 * The KV cache is updated as in dv_sparse_attn.
 */
size_t dv_sparse_block_workspace_bytes(const dv_attn *a, const dv_mlp *m, const dv_predictor *pa,
                                       const dv_predictor *pm, const dv_kv *kv, int32_t B,
                                       int32_t k_heads, int32_t k_mlp);
dv_status dv_sparse_block(const dv_attn *a, const dv_mlp *m, const dv_predictor *pa,
                          const dv_predictor *pm, const dv_ln *ln, const dv_kv *kv,
                          const float *x_in, float *x_out, int32_t B, int32_t k_heads,
                          int32_t k_mlp, int32_t mode, int32_t batch_mode, float scale,
                          int32_t *heads_out, int32_t *idx_out, void *ws, size_t ws_bytes,
                          uint32_t flags, void *stream);

/* ------------------------------------------------- several layers, look-ahead
 * dv_sparse_decode: n_layers decoder layers for one token (B = 1) with the cross-layer
 * look-ahead of Section 4.3 ("Approach"): the sets of layer l+1 are predicted from the
 * input of layer l, so the prediction needs nothing layer l computes.
 *   x_0 = LN1^0(y_0),  x_l = LN1^l(y_l)           (layer l's first layer norm)
 *   S^0     = (top-k_heads(SP_A^0(x_0)), top-k_mlp(SP_M^0(x_0)))
 *   S^{l+1} = (top-k_heads(SP_A^{l+1}(x_l)), top-k_mlp(SP_M^{l+1}(x_l)))
 *   y_{l+1} = y~ + MLP^l_{S_M^l}(LN2^l(y~)),  y~ = y_l + MHA^l_{S_A^l}(x_l)
 *   x_out   = y_{n_layers}
 * SP^j are layer j's predictors (pa, pm of layers[j], which score layer j's heads and
 * neurons). Layer l+1's predictor work runs inside layer l's launches (its first layer
 * beside the Q/K/V rows over the same staged x_l, its scores and head set in a launch
 * before the out-projection, its neuron set in the next QKV launch), so a layer costs
 * five launches and layer 0 two more. Each layer updates its own KV cache as
 * dv_sparse_attn does.
 *   layers       [n_layers] layer descriptors; every layer has layer 0's shapes and types;
 *                kv.B must be 1.
 *   heads_out    [n_layers][k_heads] or NULL: S_A^l, ascending.
 *   idx_out      [n_layers][k_mlp] or NULL: S_M^l, ascending.
 * The sets are produced inside the call, so DV_VALIDATE has nothing to check here. */
typedef struct dv_layer {
  dv_attn attn;
  dv_mlp mlp;
  dv_predictor pa, pm;   /* head predictor (n_out = H), neuron predictor (n_out = N) */
  dv_ln ln;
  dv_kv kv;
} dv_layer;

size_t dv_sparse_decode_workspace_bytes(const dv_layer *layers, int32_t n_layers, int32_t k_heads,
                                        int32_t k_mlp);
dv_status dv_sparse_decode(const dv_layer *layers, int32_t n_layers, const float *x_in, float *x_out,
                           int32_t k_heads, int32_t k_mlp, float scale, int32_t *heads_out,
                           int32_t *idx_out, void *ws, size_t ws_bytes, uint32_t flags, void *stream);

/* ------------------------------------------------- decoder layer, no allocation
 * dv_sparse_block_noalloc: for callers that cannot allocate device memory (work being
 * captured into a graph, serving loops or harnesses that forbid the allocator). The
 * same layer, arguments and results as dv_sparse_block, without a workspace: its
 * scratch space is a fixed array of DV_STATIC_SCRATCH_BYTES inside the library, one
 * per device, held until the process ends. The call allocates nothing (no hipMalloc,
 * no allocating library routine); its first call on a device looks up that device's
 * copy of the array.
 *   Limit.  A call whose dv_sparse_block_workspace_bytes exceeds DV_STATIC_SCRATCH_BYTES
 *           returns DV_ERR_WORKSPACE and enqueues nothing (batch 1 at the OPT-175B
 *           shape needs about 2.2 MB).
 *   Races.  Every call on one device uses the same array: calls that overlap in time
 *           on one device (other streams, other threads) must be ordered by the
 *           caller. Nothing in the array needs to start cleared.
 */
#define DV_STATIC_SCRATCH_BYTES (16u << 20)
dv_status dv_sparse_block_noalloc(const dv_attn *a, const dv_mlp *m, const dv_predictor *pa,
                                  const dv_predictor *pm, const dv_ln *ln, const dv_kv *kv,
                                  const float *x_in, float *x_out, int32_t B, int32_t k_heads,
                                  int32_t k_mlp, int32_t mode, int32_t batch_mode, float scale,
                                  int32_t *heads_out, int32_t *idx_out, uint32_t flags, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* DV_H */
