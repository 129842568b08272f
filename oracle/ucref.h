/*
 * ucref.h -- CPU oracle for mixed-policy KV attention (test infrastructure).
 *
 * A plain, slow, obviously-correct host implementation of what the GPU
 * library computes, written from the UniCache paper.  Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg use it; the product
 * path never does.  It shares no code, header or constant with the GPU
 * library.
 *
 * The oracle follows the paper's own reference formulation (App. E: attention
 * masks and fake quantization): evicted rows are masked out of a full-length
 * sequence and quantised rows are replaced by their dequantised values, so a
 * physically compacted / packed cache must give the same attention.
 * Floating-point attention and scoring run in IEEE double; the quantizer runs
 * in IEEE binary32 without contraction, since its codes are defined there.
 *
 * dtype codes: 0 = fp32, 1 = fp16, 2 = bf16 (stored as raw 16-bit patterns).
 */
#ifndef UCREF_H
#define UCREF_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* exact widening of n stored elements to double */
void ucref_widen(const void* x, int dtype, int64_t n, double* out);
/* value of each binary32 element after rounding to dtype (nearest even) */
void ucref_round_value(const float* x, int dtype, int64_t n, double* out);

/* Group-wise asymmetric min/max quantization (keys per channel over G rows,
 * values per row over G channels); see ucref.cpp for the definition. */
int ucref_quantize(int BH, int N, int D, int G, const int32_t* bits, int dtype,
                   const void* k, const void* v, uint8_t* codes_k,
                   uint8_t* codes_v, const int64_t* code_off, float* scale_k,
                   float* min_k, float* scale_v, float* min_v, void* tail_k,
                   void* tail_v);

/* Logical values (rounded to dtype, widened to double) of a packed segment,
 * [BH, N, D] for keys and for values. */
int ucref_dequant(int BH, int N, int D, int G, const int32_t* bits, int dtype,
                  const uint8_t* codes_k, const uint8_t* codes_v,
                  const int64_t* code_off, const float* scale_k,
                  const float* min_k, const float* scale_v, const float* min_v,
                  const void* tail_k, const void* tail_v, double* khat,
                  double* vhat);

/* Attention-probability importance (Sec. 3.3 Eq. 1 terms, summed over the
 * query heads sharing a KV head and over the observation window). */
void ucref_score(int B, int Hq, int Hkv, int D, int W, int64_t N,
                 const double* q, const double* k, const int32_t* seg_of_row,
                 int n_segs, double sm_scale, double* score, double* mass);

/* Deterministic top-k + recent selection; keep_idx ascending. */
int ucref_select(int BH, int N, const float* scores, int k, int n_recent,
                 int32_t* keep_idx);

/* Masked shared-softmax attention over the logical sequence. */
void ucref_attend(int B, int Hq, int Hkv, int D, int M, int64_t N,
                  const double* q, const double* k, const double* v,
                  const uint8_t* present, const int32_t* seg_of_row,
                  int n_segs, double sm_scale, double* o, double* lse,
                  double* seg_lse, double* seg_mass);

/* Byte accounting of one (b, h_kv) (storage budget, Sec. 3.3). */
int64_t ucref_dense_bytes(int64_t rows, int D, int dtype);
int64_t ucref_evicted_bytes(int64_t rows, int D, int dtype);
int64_t ucref_packed_bytes(int64_t N, int D, int G, int bits, int dtype);
int64_t ucref_evict_rows(double budget, double fixed, int64_t N, int D,
                         int dtype);
int ucref_assign_bits(int n_heads, const double* mass, int64_t N, int D, int G,
                      int dtype, double budget, double fixed, int32_t* bits);

/* Sec. 3.3 Eq. 2 (type budgets) and Eq. 3 (retention schedule). */
/* Sec. 3.2 / App. B: fraction of each row's score mass on its k largest
 * scores. */
int ucref_topk_mass(int BH, int N, const float* scores, int k, double* frac);

/* Sec. 3.4: index of the most faithful (bits, group) configuration at or
 * after `first` that fits the budget (see ucref.cpp). */
int ucref_quant_config(double budget, int64_t N, int D, int dtype, int n_heads, int first);
int ucref_type_budget(int n, const double* mass, const double* b_prev,
                      double B_total, double* b_next);
double ucref_retention_next(double rho, double rho_init, double rho_min,
                            double M_c, double M_0);

/* Number of OpenMP threads the oracle's parallel loops use (<= 0: default). */
int ucref_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
