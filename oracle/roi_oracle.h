/*
 * roi_oracle.h -- declarations of the plain CPU oracle of the RoI N:M mask
 * sampler ("Reservoir of Importance: Learning Semi-Structured Sparsity with
 * Differentiable Subset Sampling", arxiv 2608.23048).
 *
 * TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test suite, the
 * smoke check and the benchmark's CPU-baseline leg may load this library.
 * It shares no code, header, table or constant with the HIP library.
 *
 * Every pointer is a host pointer.  The arithmetic is scalar C; the *_mt
 * entry points only split the groups over threads.  Floating-point outputs of the relaxation
 * and of the backward are fp64; keys are fp32 because the noise definition
 * fixes them in fp32 (see roi_oracle.c).
 */
#ifndef ROI_ORACLE_H
#define ROI_ORACLE_H
#include <stdint.h>
#ifdef __cplusplus
extern "C" {
#endif

/* Noise primitives. */
void     oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);
uint32_t oracle_philox_word(uint64_t seed, uint64_t step, uint64_t elem);
float    oracle_uniform(uint32_t word);
float    oracle_log(float x);
void     oracle_log_array(const float* x, int64_t n, float* out);
float    oracle_gumbel(float u);
void     oracle_gumbel_from_words(const uint32_t* words, int64_t n, float* g);
void     oracle_keys(const float* phi, int64_t numel, float lambda, uint64_t seed, uint64_t step,
                     uint64_t elem_offset, float* kappa);

/* Group-level steps on explicit keys (for pins). */
int  oracle_topn(const float* kappa, int m, int n, uint8_t* order, uint8_t* hard);
int  oracle_relax_fwd(const double* kappa, int m, int n, double tau, double* S);
int  oracle_relax_bwd(const double* kappa, int m, int n, double tau, const double* sbar,
                      double* dkappa);

/* Whole-array forward / backward over numel elements (numel % m == 0). */
int roi_oracle_fwd(const uint16_t* W, const float* logits, int64_t numel, int n, int m,
                   float tau, float lambda, uint64_t seed, uint64_t step, uint64_t elem_offset,
                   uint16_t* W_masked, double* soft_mask, uint8_t* sel_idx);
int roi_oracle_bwd(const uint16_t* grad_W_masked, const uint16_t* W, const float* logits,
                   int64_t numel, int n, int m, float tau, float lambda, uint64_t seed,
                   uint64_t step, uint64_t elem_offset, double* grad_logits);

/* Same on gathered groups: group q holds elements [q*m, q*m+m) of the
 * gathered arrays, and its first element has global index group_elem[q]. */
int roi_oracle_fwd_groups(const uint16_t* W, const float* logits, int64_t ngroups,
                          const uint64_t* group_elem, int n, int m, float tau, float lambda,
                          uint64_t seed, uint64_t step, uint16_t* W_masked, double* soft_mask,
                          uint8_t* sel_idx);
int roi_oracle_bwd_groups(const uint16_t* grad_W_masked, const uint16_t* W, const float* logits,
                          int64_t ngroups, const uint64_t* group_elem, int n, int m, float tau,
                          float lambda, uint64_t seed, uint64_t step, double* grad_logits);

/* The whole-array forward and backward on `threads` POSIX threads (contiguous
 * ranges of groups; the same bits for any thread count), and the relaxation's
 * backward on given fp64 keys over ngroups groups of m. */
int roi_oracle_fwd_mt(const uint16_t* W, const float* logits, int64_t numel, int n, int m,
                      float tau, float lambda, uint64_t seed, uint64_t step, uint64_t elem_offset,
                      uint16_t* W_masked, double* soft_mask, uint8_t* sel_idx, int threads);
int roi_oracle_bwd_mt(const uint16_t* grad_W_masked, const uint16_t* W, const float* logits,
                      int64_t numel, int n, int m, float tau, float lambda, uint64_t seed,
                      uint64_t step, uint64_t elem_offset, double* grad_logits, int threads);
int oracle_relax_bwd_groups(const double* kappa, int64_t ngroups, int m, int n, double tau,
                            const double* sbar, double* dkappa, int threads);

/* Exponential annealing of a temperature. */
double oracle_anneal(double v_init, double v_end, double t, double t_anneal);

/* Final mask (top-n of the logits) in dense and compressed form; meta only
 * for 2:4.  Any output may be NULL. */
int oracle_export(const float* logits, const uint16_t* W, int64_t numel, int n, int m,
                  uint16_t* W_masked, uint16_t* values, uint8_t* idx, uint32_t* meta);

/* Categorical sampler (one logit per candidate mask): candidates, forward
 * (W_masked, S fp64, chosen candidate) and backward (dL/dalpha fp64). */
int oracle_cat_candidates(int n, int m, uint32_t* masks);
int oracle_cat_fwd(const uint16_t* W, const float* alpha, int64_t ngroups, int n, int m,
                   float tau, float lambda, uint64_t seed, uint64_t step, uint64_t group_offset,
                   uint16_t* W_masked, double* S, uint8_t* choice);
int oracle_cat_bwd(const uint16_t* G, const uint16_t* W, const float* alpha, int64_t ngroups,
                   int n, int m, float tau, float lambda, uint64_t seed, uint64_t step,
                   uint64_t group_offset, double* dalpha);

/* AdamW step on numel logits from an fp64 gradient (fp64 outputs). */
int oracle_adamw(const double* grad, int64_t numel, double lr, double beta1, double beta2,
                 double eps, double weight_decay, int64_t t, const float* phi, const float* m,
                 const float* v, double* phi_out, double* m_out, double* v_out);

#ifdef __cplusplus
}
#endif
#endif
