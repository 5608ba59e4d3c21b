/*
 * roi.h -- C ABI of the MI355X (gfx950) RoI differentiable N:M mask sampler.
 *
 * The method: "Reservoir of Importance: Learning Semi-Structured Sparsity with
 * Differentiable Subset Sampling" (arxiv 2608.23048).  Every group of m
 * consecutive weights carries m logits phi (one per weight, §4.2.1).  Each
 * training step perturbs them with Gumbel noise into keys (§3.2, §4.2.2),
 * keeps the n largest keys (hard Gumbel-Top-K, §3.2), and relaxes that
 * selection into a soft n-hot mask S by n softmax steps (§3.2 recursion,
 * Appendix Algorithm 1).  The forward emits the hard-masked weights; the
 * backward differentiates through the relaxation (the straight-through
 * variant of the appendix, "Comparison with Straight-Through Gumbel-Top-K").
 *
 * Conventions shared by every entry point
 * ----------------------------------------
 *  - Pointers are DEVICE pointers on the current HIP device, 16-byte aligned,
 *    contiguous; inputs and outputs must not overlap.  The caller owns all
 *    memory; the library allocates none.
 *  - bf16 tensors are passed as their raw 16-bit patterns (uint16_t).
 *  - A weight tensor is row-major [rows, cols] (PyTorch Linear: [out, in]);
 *    groups are m consecutive elements along cols, so cols % m == 0.  Any
 *    back-to-back stack of such tensors is itself a valid [1, total] input:
 *    groups never straddle tensors, and the noise depends only on the global
 *    element index.
 *  - Calls are asynchronous on `stream` (0 = the null stream).  Argument
 *    errors are detected on the host and returned before anything is
 *    launched; nothing is written then.  No exceptions cross the ABI.
 *  - Return value: ROI_OK or a negative roi_status; roi_last_error() gives a
 *    thread-local human-readable detail of the last failure.
 *  - Supported patterns: m in {4, 8, 16, 32} with 1 <= n <= m.
 *
 * Noise (the same definition the forward and the backward use):
 *  - global element index e = elem_offset + (flat index of the element);
 *  - x = word (e mod 4) of Philox4x32-10 (Salmon et al., SC'11) with key
 *    (lo32 seed, hi32 seed) and counter (lo32 e/4, hi32 e/4, lo32 step,
 *    hi32 step);
 *  - u = (2 (x >> 9) + 1) 2^-24, in (0, 1) (Algorithm 1: u ~ Uniform(0,1));
 *  - g = -L(-L(u)) with L the library's deterministic fp32 logarithm
 *    (Algorithm 1: g = -log(-log u)): x = z 2^k with z in [0.703125, 1.40625),
 *    a 128-cell table of (1/c, -ln(1/c)) (the two cells touching 1 hold
 *    (1, 0)), r = fma(z, 1/c, -1), ln(1+r) by its degree-4 series, and
 *    L = fma(k, ln2, -ln(1/c) + ln(1+r)); a fixed sequence of IEEE fp32
 *    operations, so the value is reproducible (max error 1.45 ulp);
 *  - kappa = fl(fl(phi / lambda) + g) in fp32 (§3.2 key; §4.2.3 applies the
 *    trick to phi / lambda).
 *  Given (seed, step, elem_offset) the noise is a pure function, so the
 *  backward regenerates it instead of storing it, and any split of a stack
 *  into calls with matching elem_offset gives identical results.
 */
#ifndef ROI_H
#define ROI_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    ROI_OK = 0,
    ROI_E_INVAL = -1,       /* invalid argument (sizes, pattern, temperatures, pointers) */
    ROI_E_UNSUPPORTED = -2, /* valid for the method but not built: m outside {4, 8, 16, 32} */
    ROI_E_HIP = -3          /* the HIP runtime reported an error at launch */
} roi_status;

/*
 * roi_mask_fwd -- one forward sample of the n:m mask for every group.
 *
 * §3.2 / §4.2.2: keys kappa = phi/lambda + g; hard selection = the n largest
 * keys of each group (ties go to the lower index; -0.0 and +0.0 tie).
 * §4.1: W_masked = W (.) hard mask (pruned entries are +0.0, bits 0x0000).
 * §3.2 recursion / Algorithm 1: soft_mask S = sum_{k=1..n} mu^(k) with
 * alpha^(1) = kappa, mu^(k) = softmax(alpha^(k) / tau),
 * alpha^(k+1) = alpha^(k) + log(1 - mu^(k)), computed in fp32 (log(1 - mu) is
 * floored at log(FLT_MIN)).
 *
 *  W          bf16 [rows, cols]          frozen weights (read)
 *  logits     fp32 [rows, cols]          phi (read)
 *  rows, cols sizes, rows >= 0, cols >= 0, cols % m == 0, rows * cols < 2^62
 *  n, m       keep n of every m; m in {4, 8, 16, 32}, 1 <= n <= m
 *  tau        relaxation temperature, finite, > 0 (used only for soft_mask)
 *  lambda     sampling temperature, finite, > 0 (§4.2.3)
 *  seed, step Philox key and step counter
 *  elem_offset global index of element 0; elem_offset % m == 0 (so groups of a
 *             stack keep their positions in the global index space)
 *  W_masked   bf16 [rows, cols]          (written; required)
 *  soft_mask  fp32 [rows, cols] or NULL  (written when not NULL)
 *  sel_idx    uint8 [rows*cols/m, n] or NULL: the kept indices of each group in
 *             selection order (descending key)   (written when not NULL)
 */
int roi_mask_fwd(const uint16_t* W, const float* logits, int64_t rows, int64_t cols, int n,
                 int m, float tau, float lambda, uint64_t seed, uint64_t step,
                 uint64_t elem_offset, uint16_t* W_masked, float* soft_mask, uint8_t* sel_idx,
                 hipStream_t stream);

/*
 * roi_mask_fwd_soft -- the pure soft forward (the paper's default setting:
 * "w/o STE" in the appendix comparison with the straight-through variant;
 * §4.2.2 relaxation used directly in the forward pass).  Same arguments and
 * noise as roi_mask_fwd; the output is
 *   W_soft = bf16_rne(W (.) S), S = sum_{k=1..n} mu^(k) (fp32, §3.2 recursion),
 * and soft_mask / sel_idx, when not NULL, receive S and the hard top-n indices
 * of the same keys.  The backward is roi_mask_bwd (the relaxation is the
 * differentiated path in both settings).
 * S is always evaluated at the exact keys (as in roi_mask_fwd), and W_soft is
 * the bf16 rounding of W (.) S; with soft_mask and sel_idx both NULL a kernel
 * without the selection runs, with the same W_soft bits.
 */
int roi_mask_fwd_soft(const uint16_t* W, const float* logits, int64_t rows, int64_t cols, int n,
                      int m, float tau, float lambda, uint64_t seed, uint64_t step,
                      uint64_t elem_offset, uint16_t* W_soft, float* soft_mask, uint8_t* sel_idx,
                      hipStream_t stream);

/*
 * roi_mask_bwd -- dL/dlogits from dL/dW_masked.
 *
 * Straight-through (Appendix, Comparison with Straight-Through Gumbel-Top-K):
 * the forward value is the hard mask, the backward goes through the
 * relaxation as if W_masked = W (.) S.  So dL/dS = grad_W_masked (.) W (exact
 * in fp32), dL/dkappa is the reverse-mode derivative of the §3.2 recursion,
 * and dL/dphi = dL/dkappa / lambda.  The keys are regenerated from
 * (seed, step, elem_offset) and must match the forward call's arguments: the
 * derivative is taken at exactly the fp32 keys the forward sampled.
 *
 *  grad_W_masked bf16 [rows, cols]       (read)
 *  W, logits, rows, cols, n, m, tau, lambda, seed, step, elem_offset: as in
 *             roi_mask_fwd
 *  grad_logits fp32 [rows, cols]         (overwritten)
 */
int roi_mask_bwd(const uint16_t* grad_W_masked, const uint16_t* W, const float* logits,
                 int64_t rows, int64_t cols, int n, int m, float tau, float lambda, uint64_t seed,
                 uint64_t step, uint64_t elem_offset, float* grad_logits, hipStream_t stream);

/*
 * Grouped calls: one call over many separately allocated tensors (e.g. every
 * linear layer of a model), with the shared pattern, temperatures, seed and
 * step.  Tensor i is processed exactly as the single-tensor call with its own
 * pointers, rows, cols and elem_offset would process it (same outputs, bit
 * for bit); the library launches the work of up to 32 tensor pieces per grid
 * instead of one grid per tensor.  The descriptor array is host memory, read
 * during the call only; the pointers in it follow the conventions above.
 * Tensors with rows * cols == 0 are skipped (their pointers may be NULL).
 * soft_mask and sel_idx must each be non-NULL for every nonempty tensor or
 * for none.  No output may overlap any input or output of any tensor (inputs
 * may overlap each other).  Any argument error returns before anything is
 * launched; roi_last_error() names the offending tensor.
 */
typedef struct {
    const uint16_t* W;     /* bf16 [rows, cols] (read) */
    const float* logits;   /* fp32 [rows, cols] (read) */
    uint16_t* W_masked;    /* bf16 [rows, cols] (written) */
    float* soft_mask;      /* fp32 [rows, cols] or NULL */
    uint8_t* sel_idx;      /* uint8 [rows*cols/m, n] or NULL */
    int64_t rows, cols;
    uint64_t elem_offset;  /* global index of element 0, % m == 0 */
} roi_fwd_tensor;

typedef struct {
    const uint16_t* grad_W_masked; /* bf16 [rows, cols] (read) */
    const uint16_t* W;             /* bf16 [rows, cols] (read) */
    const float* logits;           /* fp32 [rows, cols] (read) */
    float* grad_logits;            /* fp32 [rows, cols] (overwritten) */
    int64_t rows, cols;
    uint64_t elem_offset;
} roi_bwd_tensor;

/* roi_mask_fwd over `count` tensors (count >= 0). */
int roi_mask_fwd_grouped(const roi_fwd_tensor* tensors, int count, int n, int m, float tau,
                         float lambda, uint64_t seed, uint64_t step, hipStream_t stream);
/* roi_mask_fwd_soft over `count` tensors (W_masked receives W_soft). */
int roi_mask_fwd_soft_grouped(const roi_fwd_tensor* tensors, int count, int n, int m, float tau,
                              float lambda, uint64_t seed, uint64_t step, hipStream_t stream);
/* roi_mask_bwd over `count` tensors. */
int roi_mask_bwd_grouped(const roi_bwd_tensor* tensors, int count, int n, int m, float tau,
                         float lambda, uint64_t seed, uint64_t step, hipStream_t stream);

/*
 * roi_mask_bwd_adamw -- roi_mask_bwd with one AdamW step on the logits fused
 * in (appendix: the logits are trained with AdamW, beta1 = 0.9, beta2 = 0.95,
 * weight decay 0.05, a learning rate decaying from 1e-3 to 1e-4; the weights
 * stay frozen).  With g = dL/dlogits of this step, every logit becomes
 *   phi' = phi (1 - lr wd) - (lr / (1 - beta1^t)) m' / (sqrt(v' / (1 - beta2^t)) + eps),
 *   m'   = beta1 m + (1 - beta1) g,   v' = beta2 v + (1 - beta2) g^2
 * (decoupled weight decay, Loshchilov & Hutter; bias-corrected moments,
 * Kingma & Ba), in fp32.  The keys use the logits as they were before the
 * step.  The gradient is never stored unless grad_logits is given, so the
 * step moves 28 bytes per weight instead of 12 (backward) + 28 (optimizer).
 *
 *  logits      fp32 [rows, cols]  read, then overwritten with phi'
 *  exp_avg     fp32 [rows, cols]  m, overwritten with m'
 *  exp_avg_sq  fp32 [rows, cols]  v, overwritten with v'
 *  grad_logits fp32 [rows, cols]  or NULL: also written with g
 *  opt         host struct: lr >= 0, 0 <= beta1, beta2 < 1, eps > 0,
 *              weight_decay >= 0 (all finite), t >= 1 = this step's 1-based
 *              optimizer step count; the caller schedules lr (e.g. with
 *              roi_anneal).
 *  Other arguments as in roi_mask_bwd.  The moments and grad_logits must not
 *  overlap each other, the logits or the inputs.
 */
typedef struct {
    float lr;
    float beta1, beta2;
    float eps;
    float weight_decay;
    int64_t t;
} roi_adamw_params;

int roi_mask_bwd_adamw(const uint16_t* grad_W_masked, const uint16_t* W, float* logits,
                       float* exp_avg, float* exp_avg_sq, float* grad_logits, int64_t rows,
                       int64_t cols, int n, int m, float tau, float lambda, uint64_t seed,
                       uint64_t step, uint64_t elem_offset, const roi_adamw_params* opt,
                       hipStream_t stream);

/* roi_mask_bwd_adamw over `count` tensors (grouped-call conventions above). */
typedef struct {
    const uint16_t* grad_W_masked; /* bf16 [rows, cols] (read) */
    const uint16_t* W;             /* bf16 [rows, cols] (read) */
    float* logits;                 /* fp32 [rows, cols] (read, overwritten) */
    float* exp_avg;                /* fp32 [rows, cols] (read, overwritten) */
    float* exp_avg_sq;             /* fp32 [rows, cols] (read, overwritten) */
    float* grad_logits;            /* fp32 [rows, cols] or NULL */
    int64_t rows, cols;
    uint64_t elem_offset;
} roi_adamw_tensor;

int roi_mask_bwd_adamw_grouped(const roi_adamw_tensor* tensors, int count, int n, int m,
                               float tau, float lambda, uint64_t seed, uint64_t step,
                               const roi_adamw_params* opt, hipStream_t stream);

/*
 * roi_mask_export -- the final mask after training, in dense and compressed
 * form.  §4.2.3 anneals the sampling temperature lambda towards 0; the
 * sampler's lambda -> 0 limit keeps the n largest logits of each group (ties
 * to the lower index, as in the sampler), with no noise.  This call writes
 * that mask:
 *  W_masked bf16 [rows, cols] or NULL: W where kept, +0.0 elsewhere;
 *  values   bf16 [rows*cols/m, n] or NULL: the kept weights of each group in
 *           increasing index order (the compressed sparse weight);
 *  idx      uint8 [rows*cols/m, n] or NULL: their indices, increasing;
 *  meta     uint32 [ceil(rows*cols/m / 8)] or NULL, 2:4 only: group q's two
 *           indices as 2-bit fields in bits 4(q%8) .. 4(q%8)+3 of word q/8,
 *           the lower index in the low two bits (the index metadata that
 *           accompanies 2:4-compressed values).
 * At least one output must be requested.  W may be NULL when only idx and
 * meta are.  logits, W, rows, cols, n, m as in roi_mask_fwd (no temperatures,
 * seed or step).
 */
int roi_mask_export(const float* logits, const uint16_t* W, int64_t rows, int64_t cols, int n,
                    int m, uint16_t* W_masked, uint16_t* values, uint8_t* idx, uint32_t* meta,
                    hipStream_t stream);

/*
 * The categorical mask sampler: the parameterization the paper compares with
 * (appendix, "Optimization Efficiency"), one logit per feasible n-hot mask of
 * a group, Pr(c) = softmax(alpha)_c, sampled with Gumbel-Softmax.  It is a
 * second workload on the same harness: binom(m, n) logits per group instead
 * of m (1.5x the weights at 2:4, 3.5x at 2:8, 8.75x at 4:8).
 *  - candidates: the n-subsets of {0..m-1} in lexicographic order;
 *  - keys kappa_c = fl(fl(alpha_c / lambda) + g_c), g_c the noise of element
 *    4 B Q + c with B = ceil(C / 4), Q = group_offset + local group index;
 *  - hard sample: the candidate of largest key (ties to the lower candidate),
 *    W_masked = W (.) its mask, choice = its index;
 *  - soft mask S_j = sum_c softmax(kappa / tau)_c [j in c];
 *  - backward (straight-through): ybar_c = sum_{j in c} (dL/dW_masked (.) W)_j,
 *    dL/dalpha = softmax (.) (ybar - <softmax, ybar>) / (tau lambda).
 * m in {4, 8}.  cat_logits fp32 [rows*cols/m, C] (group-major).  Other
 * arguments and conventions as for the item sampler.
 */
/* binom(m, n), the logits per group, or -1 for an unsupported pattern. */
int roi_cat_num_candidates(int n, int m);
int roi_cat_mask_fwd(const uint16_t* W, const float* cat_logits, int64_t rows, int64_t cols,
                     int n, int m, float tau, float lambda, uint64_t seed, uint64_t step,
                     uint64_t group_offset, uint16_t* W_masked, float* soft_mask,
                     uint8_t* choice, hipStream_t stream);
int roi_cat_mask_bwd(const uint16_t* grad_W_masked, const uint16_t* W, const float* cat_logits,
                     int64_t rows, int64_t cols, int n, int m, float tau, float lambda,
                     uint64_t seed, uint64_t step, uint64_t group_offset, float* grad_cat_logits,
                     hipStream_t stream);

/*
 * roi_gumbel_noise -- the noise of `count` consecutive elements starting at
 * global index elem_offset (elem_offset % 4 == 0): the raw Philox words
 * and/or g = -L(-L(u)) (Algorithm 1).  Either output may be NULL, not both.
 *  words  uint32 [count] or NULL; gumbel fp32 [count] or NULL
 */
int roi_gumbel_noise(uint64_t seed, uint64_t step, uint64_t elem_offset, int64_t count,
                     uint32_t* words, float* gumbel, hipStream_t stream);

/*
 * roi_gumbel_from_words -- g = -L(-L(u(x))) for caller-given 32-bit words x
 * (Algorithm 1 applied to explicit uniforms; exposes the deterministic noise
 * transform on its own).  words uint32 [count] (read), gumbel fp32 [count]
 * (written).
 */
int roi_gumbel_from_words(const uint32_t* words, int64_t count, float* gumbel,
                          hipStream_t stream);

/*
 * roi_fast_noise_from_words -- the noise in log2 units from the hardware
 * logarithm, K(x) = -log2(-log2 u(x)) = g log2(e) + log2(ln 2) up to a few
 * ulp: the form the straight-through forwards use for their key comparisons,
 * falling back to the exact keys whenever two keys are closer than the proven
 * bound of this form's error (no relaxation uses it).  words uint32 [count]
 * (read), out fp32 [count] (written).
 */
int roi_fast_noise_from_words(const uint32_t* words, int64_t count, float* out, hipStream_t stream);

/*
 * roi_anneal -- §4.2.3 exponential annealing, host-side:
 * v_t = max{ v_end, v_init (v_end / v_init)^(t / t_anneal) }, evaluated in
 * fp64 and rounded to fp32.  Requires v_init > 0, v_end > 0, t >= 0,
 * t_anneal > 0; returns NaN otherwise.
 */
float roi_anneal(float v_init, float v_end, int64_t t, int64_t t_anneal);

/*
 * roi_stream_copy -- not part of the method: a plain copy of nbytes from src
 * to dst (device pointers, 16-byte aligned, not overlapping; nbytes a
 * multiple of 16), with the sampler kernels' access pattern: 16 bytes per
 * lane, non-temporal loads and stores, one pass of a one-shot grid.  The
 * benchmark times it as the same GPU's achievable streaming bandwidth.
 * Asynchronous on stream; ROI_E_INVAL for bad arguments before any launch.
 */
int roi_stream_copy(const void* src, void* dst, int64_t nbytes, hipStream_t stream);

/* Static description of a status code. */
const char* roi_status_string(int status);
/* Thread-local detail of the last failed call on this thread ("" if none). */
const char* roi_last_error(void);
/* ABI version, currently 1. */
int roi_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* ROI_H */
