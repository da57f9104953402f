/*
 * ckm_ref -- CPU oracle for batched evaluation of rounded rematerialization
 * schedules (Checkmate, Jain et al., MLSys 2020: Sections 4.1-4.6, 5.1-5.3,
 * Algorithm 2).
 *
 * TEST INFRASTRUCTURE ONLY. This is a plain, single-threaded, deliberately
 * slow C implementation of the definitions, used to check the GPU library.
 * Only the test suite, the smoke entry point and the benchmark's CPU-baseline
 * leg may load it. It shares no code with the GPU library.
 *
 * Conventions (0-indexed form of the paper's 1-indexed notation):
 *   nodes and stages are 0..n-1; node t is computed for the first time in
 *   stage t (frontier-advancing stages, Section 4.6);
 *   S[t][i] = 1: value i is resident at the start of stage t (only i < t);
 *   R[t][i] = 1: node i is (re)computed during stage t (only i <= t);
 *   byte matrices are n*n row-major, S[t*n + i];
 *   S[n][.] (one past the last stage) is all zero: nothing is kept after
 *   the final stage.
 *
 * Parity pins: see the test suite. The Philox4x32-10 bit stream has no
 * offline known-answer vectors here ("parity unpinned" for the raw RNG
 * bits); it is checked by statistics of the rounding it drives and by an
 * independent implementation of the same published definition.
 */
#ifndef CKM_REF_H
#define CKM_REF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  CKM_REF_OK = 0,
  CKM_REF_E_INVALID_ARG = 1,
  CKM_REF_E_GRAPH = 2,
  CKM_REF_E_OVERFLOW = 3
};

enum { CKM_REF_F_DET0 = 1u };

/* Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC'11). */
void ckm_ref_philox4x32_10(const uint32_t key[2], const uint32_t ctr[4], uint32_t out[4]);

/* The 16-bit uniform draw u_{k,t,i}: key = seed (low word, high word),
 * counter = (i / 8, t, k, 0), draw = 16-bit half (i mod 8) of the 128-bit
 * output, low half of word 0 first. */
uint32_t ckm_ref_draw(uint64_t seed, uint32_t k, uint32_t t, uint32_t i);

/* Graph validation: topological numbering (every dep i of j has i < j),
 * no duplicate deps, non-negative sizes and costs, and no int64 overflow of
 * M_in + 2 M_param + sum(M) or of n * sum(C). Returns a CKM_REF_* code. */
int ckm_ref_validate_graph(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                           const int64_t* cost, const int64_t* size,
                           int64_t m_input, int64_t m_param);

/* Thresholds q[t][i] = floor(clamp(S*[t][i], 0, 1) * 65536) for i < t, 0
 * elsewhere; q is n*n row-major. Returns CKM_REF_E_INVALID_ARG if an i < t
 * entry of S* is NaN. */
int ckm_ref_quantize(int32_t n, const double* s_frac, int64_t ld, uint32_t* q);

/* Randomized rounding of S* (Section 5.1): S[t][i] = [u_{k,t,i} < q[t][i]]. */
void ckm_ref_round_random(int32_t n, const uint32_t* q, uint64_t seed, uint32_t k, uint8_t* S);

/* Deterministic rounding of Algorithm 2: S[t][i] = [S*[t][i] > 0.5]. */
void ckm_ref_round_det(int32_t n, const double* s_frac, int64_t ld, uint8_t* S);

/* Deterministic rounding at threshold p: S[t][i] = [clamp(S*[t][i], 0, 1) > p]
 * for i < t (Section 5.1 with the strict comparison of Algorithm 2). Returns
 * CKM_REF_E_INVALID_ARG for a NaN p or a NaN S* entry with i < t. */
int ckm_ref_round_threshold(int32_t n, const double* s_frac, int64_t ld, double p, uint8_t* S);

/* Two-phase rounding's R (Section 5.2): per stage, the least set holding
 * node t (4a) and the values kept into t+1 but not held in t (1c), closed
 * under taking an operand of a computed node that stage t does not hold
 * (1b). Found by a worklist search over the dependency edges. */
void ckm_ref_solve_R(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                     const uint8_t* S, uint8_t* R);

/* Memory and cost of a schedule (Section 4.3 objective, Section 4.4 U
 * recurrence with the FREE product evaluated literally).
 * peak = max over t,k of U_{t,k}; total_cost = sum_t sum_i C_i R[t][i].
 * Optional outputs (may be NULL): stage_peak[n]; max_frees = the largest
 * number of times one value is freed within one stage (Theorem 4.1 says <= 1);
 * U_end[n] = memory in use at the end of each stage. */
void ckm_ref_simulate(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                      const int64_t* cost, const int64_t* size, int64_t m_input, int64_t m_param,
                      const uint8_t* S, const uint8_t* R, int64_t* peak, int64_t* total_cost,
                      int64_t* stage_peak, int32_t* max_frees, int64_t* U_end);

/* One candidate: round (random, or deterministic for k = 0 under DET0), solve
 * R, simulate. S_out / R_out (n*n bytes) may be NULL. */
int ckm_ref_eval_candidate(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                           const int64_t* cost, const int64_t* size, int64_t m_input,
                           int64_t m_param, const double* s_frac, int64_t ld, const uint32_t* q,
                           uint64_t seed, uint32_t k, uint32_t flags, int64_t* peak,
                           int64_t* total_cost, uint8_t* S_out, uint8_t* R_out);

/* The whole batched path: K candidates, per-candidate peak / cost / feasible
 * (peak <= budget), best_k = lexicographic minimum of (cost, peak, k) over
 * feasible candidates or -1, and the best candidate's S and R as bit rows
 * (W = ceil(n/64) uint64 words per row, bit i%64 of word i/64), zero when
 * best_k = -1. best_S / best_R may be NULL. */
int ckm_ref_round_eval(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                       const int64_t* cost, const int64_t* size, int64_t m_input, int64_t m_param,
                       const double* s_frac, int64_t ld, int32_t K, uint64_t seed, int64_t budget,
                       uint32_t flags, int64_t* peak, int64_t* total_cost, uint8_t* feasible,
                       int32_t* best_k, uint64_t* best_S, uint64_t* best_R);

/* Whether (S, R) meets what the plan generator needs: R[t][t] = 1 (4a), no
 * value both kept and recomputed in a stage, constraints (1b) and (1c).
 * Entries of S with i >= t and of R with i > t are not read. */
int ckm_ref_check_schedule(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                           const uint8_t* S, const uint8_t* R);

/* The execution plan of Section 4.9 for (S, R) as statements (op, node,
 * register, stage), op 0 = compute, 1 = deallocate, with the memory in use
 * after each statement (mem may be NULL). Each value is released after the
 * compute of the node where its FREE term (eq. collectable) is 1; releases
 * at one node go in increasing value order. Unused checkpoints
 * that are not kept are deallocated at the end of their stage, or at its
 * start when early != 0. Writes at most capacity statements; *count = the
 * plan's length. CKM_REF_E_INVALID_ARG if (S, R) fails the check above. */
int ckm_ref_plan(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx, const int64_t* size,
                 int64_t m_input, int64_t m_param, const uint8_t* S, const uint8_t* R, int early,
                 int32_t* stmts, int64_t* mem, int64_t capacity, int64_t* count);

/* Largest batch multiplier B of a schedule: sizes B * M_i (M_input, M_param
 * unscaled), peak <= budget, and the schedule's cost <= cost_cap (eq.
 * cost_constr). Searched over the simulator (doubling, then bisection); 0 if
 * B = 1 fails, `limit` if B = limit fits. */
int64_t ckm_ref_max_batch(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx, const int64_t* cost,
                          const int64_t* size, int64_t m_input, int64_t m_param, const uint8_t* S,
                          const uint8_t* R, int64_t budget, int64_t cost_cap, int64_t limit);

#ifdef __cplusplus
}
#endif
#endif
