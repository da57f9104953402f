/*
 * ckm.h -- batched evaluation of rounded rematerialization schedules on
 * MI355X (gfx950).
 *
 * The method is the approximation path of Checkmate (Jain et al., "Checkmate:
 * Breaking the Memory Wall with Optimal Tensor Rematerialization", MLSys
 * 2020): a fractional checkpoint matrix S* (the LP relaxation of Section 5.1)
 * is rounded into K candidate checkpoint matrices by randomized rounding
 * (Section 5.1); for each candidate the recomputation matrix R is repaired by
 * two-phase rounding (Algorithm 2, Section 5.2); each candidate is simulated
 * for peak memory (the U recurrence with the FREE terms, Section 4.4) and for
 * cost (the objective of Section 4.3); the cheapest candidate within the
 * memory budget (constraint U_{t,k} <= M_budget of Section 4.7) is returned.
 *
 * Index convention: nodes and stages are 0..n-1 (the paper counts from 1);
 * node t is computed for the first time in stage t (frontier-advancing
 * stages, Section 4.6). S[t][i] = 1 means value i is resident at the start of
 * stage t (only i < t); R[t][i] = 1 means node i is computed in stage t (only
 * i <= t). Nothing is kept after the last stage.
 *
 * Rounding: q[t][i] = floor(clamp(S*[t][i], 0, 1) * 65536) and candidate k
 * keeps value i into stage t iff u_{k,t,i} < q[t][i], where u is a 16-bit
 * draw of Philox4x32-10 (Salmon et al., SC'11) with key = seed (low 32 bits,
 * high 32 bits) and counter = (i / 8, t, k, 0); draw i uses 16-bit half
 * (i mod 8) of the 128-bit output, low half of word 0 first. With CKM_F_DET0
 * candidate 0 instead uses Algorithm 2's deterministic rounding S* > 0.5.
 *
 * Bit rows: a row of an n x n 0/1 matrix is W = ceil(n/64) uint64 words;
 * node i is bit (i % 64) of word (i / 64); unused high bits are zero.
 *
 * Errors never cross the ABI as exceptions: every call returns a ckm_status;
 * ckm_last_error() gives a thread-local message for the last non-OK status
 * of the calling thread. On a non-OK return the outputs are unspecified.
 *
 * Exact-arithmetic range: every memory level and cost the method forms is
 * at most M_in + 2 M_param + sum(M), or n * sum(C); a graph for which either
 * exceeds INT64_MAX is rejected with CKM_E_OVERFLOW, and every other graph is
 * evaluated exactly. (The kernels sum in IEEE binary64 while all sums stay
 * below 2^53, where it is exact, and in int64 otherwise.)
 */
#ifndef CKM_H
#define CKM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ckm_graph ckm_graph; /* opaque, immutable after creation */

typedef enum {
  CKM_OK = 0,
  CKM_E_INVALID_ARG = 1, /* bad argument: NULL, K < 1, ld < n, negative budget, NaN in S* */
  CKM_E_GRAPH = 2,       /* not topologically numbered, duplicate edge, users != transpose */
  CKM_E_OVERFLOW = 3,    /* M_in + 2 M_param + sum(M) or n * sum(C) exceeds INT64_MAX */
  CKM_E_UNSUPPORTED = 4, /* n > CKM_MAX_NODES, K > CKM_MAX_CANDIDATES (CKM_MAX_THRESHOLDS) */
  CKM_E_NOMEM = 5,       /* host or device allocation failed */
  CKM_E_DEVICE = 6       /* a HIP runtime call failed (message has the HIP error) */
} ckm_status;

enum {
  CKM_F_DET0 = 1u,    /* candidate 0 = deterministic rounding S* > 0.5 (Algorithm 2) */
  CKM_F_ROUNDED = 2u  /* ckm_evaluate_async / ckm_select_async only: ckm_round_async has
                         rounded the rows (same K, seed, CKM_F_DET0) on this work buffer */
};

#define CKM_MAX_NODES 4096
#define CKM_MAX_CANDIDATES (1 << 24)
#define CKM_MAX_THRESHOLDS (1 << 16) /* candidates of the threshold family */

/* Build a graph (Section 4.1: a DAG numbered in topological order, node v
 * with output size M_v = bytes[v] and cost C_v = cost[v]) and upload it to
 * the current HIP device.
 *   n                  number of nodes, 1..CKM_MAX_NODES
 *   dep_ptr, dep_idx   CSR of Deps: the deps of node j are
 *                      dep_idx[dep_ptr[j] .. dep_ptr[j+1]), any order, each
 *                      i < j, no duplicates; dep_ptr has n+1 entries,
 *                      dep_ptr[0] = 0
 *   user_ptr, user_idx CSR of Users (Section 4.4), or both NULL to derive it;
 *                      if given it must be the transpose of Deps
 *   cost, bytes        int64 [n], >= 0
 *   m_input, m_param   M_in and M_param of eq. U_init, >= 0
 *   out                receives the handle
 * All arrays are host arrays, copied; the caller keeps ownership.
 * Errors: CKM_E_GRAPH for a malformed CSR (dep_ptr[0] != 0, dep_ptr
 * decreasing, more than n(n-1)/2 edges), an edge i -> j with i < 0 or
 * i >= j, a duplicate edge, or Users that differ from the transpose of Deps;
 * CKM_E_OVERFLOW when M_in + 2 M_param + sum(M) or n * sum(C) exceeds
 * INT64_MAX; CKM_E_INVALID_ARG for NULL arrays or negative
 * sizes and costs; CKM_E_NOMEM, CKM_E_DEVICE when allocation or upload
 * fails. On error *out is NULL. */
ckm_status ckm_graph_create(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                            const int32_t* user_ptr, const int32_t* user_idx,
                            const int64_t* cost, const int64_t* bytes, int64_t m_input,
                            int64_t m_param, ckm_graph** out);

/* Free a graph and its device memory. NULL is ignored. The graph must not be
 * in use by work still queued on a stream, or by a synchronous call.
 *
 * Synchronous calls (ckm_round_eval, ckm_eval_schedules, ckm_threshold_eval,
 * ckm_plan, ckm_max_batch) keep a stream, device memory and pinned host
 * memory on the graph, sized by the largest call so far, and reuse them, so
 * that repeated calls allocate nothing; ckm_graph_destroy frees them. They
 * may run concurrently on one graph: a call that finds them in use by
 * another thread allocates its own for its duration. */
void ckm_graph_destroy(ckm_graph* g);

/* Number of nodes, or -1 for NULL. */
int32_t ckm_graph_num_nodes(const ckm_graph* g);

/* The whole path, synchronous, host arrays.
 *   s_frac      host float64, n rows of stride ld (ld >= n); only the
 *               strict lower triangle (i < t) is read; values are clamped
 *               to [0, 1]; NaN there gives CKM_E_INVALID_ARG
 *   K           number of candidates, 1..CKM_MAX_CANDIDATES
 *   seed        Philox key
 *   budget      M_budget in bytes, >= 0; candidate k is feasible iff its
 *               peak memory <= budget
 *   flags       0 or CKM_F_DET0
 *   peak, cost  int64 [K]: max_{t,k} U_{t,k} and sum_t sum_i C_i R[t][i]
 *   feasible    uint8 [K]: 1 iff peak <= budget
 *   best_k      lexicographic minimum of (cost, peak, k) over feasible
 *               candidates, or -1 when none is feasible
 *   best_S, best_R  uint64 [n * W] bit rows of the best candidate (zero when
 *               best_k = -1); either may be NULL
 * Runs on the current HIP device (the graph's) on an internal stream and
 * returns when the results are in the caller's arrays. */
ckm_status ckm_round_eval(const ckm_graph* g, const double* s_frac, int64_t ld, int32_t K,
                          uint64_t seed, int64_t budget, uint32_t flags, int64_t* peak,
                          int64_t* cost, uint8_t* feasible, int32_t* best_k, uint64_t* best_S,
                          uint64_t* best_R);

/* ---- asynchronous, device-pointer form --------------------------------
 * Every pointer below is device memory on the graph's device; `stream` is a
 * hipStream_t (NULL = the null stream). Calls only enqueue work; buffers must
 * stay alive until the stream has executed it. Work buffers are caller-owned
 * and sized by ckm_workspace_size; one work buffer must not be used by two
 * calls that may run concurrently. The three stages run in the order
 * quantize -> evaluate -> select, on one work buffer. The library cannot
 * check sizes behind a pointer: each array must hold the elements stated
 * for it (work_bytes is checked against the layout).
 *
 * The calls enqueue kernel launches only (no allocation, memset, copy or
 * synchronization), so a sequence of them can be captured into a HIP graph
 * on `stream` and replayed; scalar arguments (K, seed, budget, flags) are
 * fixed at capture. On a graph whose evaluate LDS holds to a few waves per
 * CU (the seen path of large graphs), an evaluate with 8 or more groups of
 * 64 candidates runs the later groups on the graph's second stream, forked
 * from `stream` and joined back to it by events before the call's work on
 * `stream` ends; a capture takes that fork and join in as dependencies. */

/* Bytes of work buffer for K candidates on graph g. This includes, when the
 * S rows of all K candidates fit in 8 GiB, room for them and for their R
 * rows (the row arrays, twice the S rows' size; 8.3 GB at n = 4001,
 * K = 4096):
 * the evaluate stage then streams each row from there instead of making it
 * twice (randomized rounding, threshold rounding) or reading it from each
 * candidate's own matrix (supplied schedules). A smaller buffer of at least
 * ckm_workspace_size_min bytes is accepted, and the rows are then made
 * inside the evaluate stage (same results). */
ckm_status ckm_workspace_size(const ckm_graph* g, int32_t K, size_t* bytes);

/* The smallest work buffer accepted for K candidates: without the row array. */
ckm_status ckm_workspace_size_min(const ckm_graph* g, int32_t K, size_t* bytes);

/* Stage a1: thresholds q (Section 5.1) and the deterministic-rounding bits of
 * Algorithm 2 from S* (device float64, n rows of stride ld >= n). A NaN in
 * the strict lower triangle is recorded in the work buffer and reported by
 * ckm_select_async through d_status. */
ckm_status ckm_quantize_async(const ckm_graph* g, const double* d_s_frac, int64_t ld,
                              void* d_work, size_t work_bytes, void* stream);

/* Stage a2 on its own: rounds every candidate's S rows (Section 5.1) once
 * into the work buffer's row array, after ckm_quantize_async. It does
 * nothing when the buffer or the problem has no room for them (see
 * ckm_workspace_size); ckm_evaluate_async then rounds inside. flags: 0 or
 * CKM_F_DET0. Call ckm_evaluate_async with CKM_F_ROUNDED and the same K,
 * seed and CKM_F_DET0 to use the rows; without CKM_F_ROUNDED it rounds them
 * again itself. */
ckm_status ckm_round_async(const ckm_graph* g, int32_t K, uint64_t seed, uint32_t flags, void* d_work,
                           size_t work_bytes, void* stream);

/* Stages a2-a5 for candidates 0..K-1: rounding, Algorithm 2's R repair,
 * memory simulation and cost. Leaves each candidate's peak and cost in the
 * work buffer (reset at the start of every call). stage_splits = number of
 * stage ranges each group of 64 candidates is split into, 1..n (0 =
 * automatic: ranges cut and ordered for load balance); results do not depend
 * on it. flags: CKM_F_DET0, and CKM_F_ROUNDED when ckm_round_async has
 * rounded the rows (with the same K, seed and CKM_F_DET0) since the last
 * ckm_quantize_async on this buffer; the rows are then not rounded again. */
ckm_status ckm_evaluate_async(const ckm_graph* g, int32_t K, uint64_t seed, uint32_t flags,
                              int32_t stage_splits, void* d_work, size_t work_bytes, void* stream);

/* Stages a6-a7: per-candidate peak / cost / feasible, the argmin, and the
 * best candidate's S and R bit rows (d_best_S / d_best_R may be NULL).
 * d_status (may be NULL) receives CKM_OK, or CKM_E_INVALID_ARG when S*
 * held a NaN (then every other output is unspecified). K, seed and flags
 * must be those given to ckm_evaluate_async. */
ckm_status ckm_select_async(const ckm_graph* g, int32_t K, uint64_t seed, int64_t budget,
                            uint32_t flags, int64_t* d_peak, int64_t* d_cost,
                            uint8_t* d_feasible, int32_t* d_best_k, uint64_t* d_best_S,
                            uint64_t* d_best_R, int32_t* d_status, void* d_work,
                            size_t work_bytes, void* stream);

/* The three stages in one call (same arguments as ckm_round_eval, all
 * arrays on the device, plus d_status, the work buffer and the stream). */
ckm_status ckm_round_eval_async(const ckm_graph* g, const double* d_s_frac, int64_t ld,
                                int32_t K, uint64_t seed, int64_t budget, uint32_t flags,
                                int64_t* d_peak, int64_t* d_cost, uint8_t* d_feasible,
                                int32_t* d_best_k, uint64_t* d_best_S, uint64_t* d_best_R,
                                int32_t* d_status, void* d_work, size_t work_bytes, void* stream);

/* ---- caller-supplied schedules -----------------------------------------
 * Evaluates K given integral checkpoint matrices S_0 .. S_{K-1} the way the
 * rounded candidates are evaluated: R by Algorithm 2's repair (Section 5.2),
 * memory by the U recurrence with the FREE terms (Section 4.4), cost by the
 * objective of Section 4.3, feasibility by peak <= budget (the U <= M_budget
 * constraint of the complete MILP, Section 4.7), and the lexicographic
 * minimum of (cost, peak, k) over feasible k (-1 if none).
 *
 * S: K matrices of n bit rows; a row is ceil(n/64) uint64 words, least
 * significant bit first: S_k[t][i] is bit i % 64 of word i / 64 of row t of
 * matrix k (the layout of best_S). Bits on or above the diagonal (i >= t)
 * are ignored. peak, cost, feasible: [K]. best_R (may be NULL): the chosen
 * matrix's R rows in the same layout, zero when best_k = -1. The
 * synchronous form takes host arrays; the asynchronous form device arrays, a
 * work buffer sized by ckm_workspace_size(g, K) and a stream, and writes
 * CKM_OK to d_status (may be NULL). */
ckm_status ckm_eval_schedules(const ckm_graph* g, const uint64_t* S, int32_t K, int64_t budget,
                              int64_t* peak, int64_t* cost, uint8_t* feasible, int32_t* best_k,
                              uint64_t* best_R);
ckm_status ckm_eval_schedules_async(const ckm_graph* g, const uint64_t* d_S, int32_t K, int64_t budget,
                                    int64_t* d_peak, int64_t* d_cost, uint8_t* d_feasible,
                                    int32_t* d_best_k, uint64_t* d_best_R, int32_t* d_status,
                                    void* d_work, size_t work_bytes, void* stream);

/* ---- threshold family --------------------------------------------------
 * One deterministic candidate per threshold: S_k[t][i] = [clamp(S*[t][i], 0,
 * 1) > p_k] for i < t, compared in double (Section 5.1's deterministic
 * rounding at a chosen threshold; Algorithm 2's is p = 0.5 with the strict
 * comparison used here). The candidates are then evaluated as the rounded
 * ones: Algorithm 2's R repair (Section 5.2), memory and cost (Sections 4.4
 * and 4.3), feasibility and the lexicographic argmin of (cost, peak, k).
 *
 * s_frac, ld: as for ckm_round_eval. p: float64 [K] thresholds, any order,
 * duplicates allowed (each is its own candidate). K: 1..CKM_MAX_THRESHOLDS.
 * A NaN threshold or a NaN in the strict lower triangle of S* gives
 * CKM_E_INVALID_ARG (the asynchronous form reports it through d_status).
 * Outputs as for ckm_round_eval; best_S and best_R may be NULL. The
 * asynchronous form takes device arrays, a work buffer sized by
 * ckm_workspace_size(g, K) and a stream. */
ckm_status ckm_threshold_eval(const ckm_graph* g, const double* s_frac, int64_t ld, const double* p,
                              int32_t K, int64_t budget, int64_t* peak, int64_t* cost, uint8_t* feasible,
                              int32_t* best_k, uint64_t* best_S, uint64_t* best_R);
ckm_status ckm_threshold_eval_async(const ckm_graph* g, const double* d_s_frac, int64_t ld, const double* d_p,
                                   int32_t K, int64_t budget, int64_t* d_peak, int64_t* d_cost,
                                   uint8_t* d_feasible, int32_t* d_best_k, uint64_t* d_best_S,
                                   uint64_t* d_best_R, int32_t* d_status, void* d_work, size_t work_bytes,
                                   void* stream);

/* ---- largest batch ------------------------------------------------------
 * The maximum-batch experiment of the evaluation: a batch multiplier B
 * scales every node size to B * M_i (M_in and M_param stay). Costs do not
 * scale. For each rounded candidate k (randomized rounding of S*, Section
 * 5.1, repaired by Algorithm 2 and simulated as in ckm_round_eval), batch[k]
 * is the largest B with peak memory <= budget. That is
 * floor((budget - base) / (peak_k - base)), base = M_in + 2 M_param, since
 * every other U term scales with B. The candidate's cost must also be
 * <= cost_cap (eq. cost_constr: at most one extra forward pass; the caller
 * computes it, 2 sum_fwd C_i + sum_bwd C_i). Otherwise batch[k] = 0. A
 * candidate with no activation bytes gets INT64_MAX. best_k: the largest B,
 * then the lexicographic minimum of (cost, peak, k); -1 when every B is 0.
 * best_batch (may be NULL) receives its B. The synchronous form takes S*
 * like ckm_round_eval. The asynchronous form reads the per-candidate totals
 * that the last ckm_evaluate_async left in the work buffer (after
 * ckm_quantize_async; K must match), so it can run beside ckm_select_async.
 * It writes the S* NaN status to d_status (may be NULL). */
ckm_status ckm_max_batch(const ckm_graph* g, const double* s_frac, int64_t ld, int32_t K, uint64_t seed,
                         uint32_t flags, int64_t budget, int64_t cost_cap, int64_t* batch, int32_t* best_k,
                         int64_t* best_batch);
ckm_status ckm_max_batch_async(const ckm_graph* g, int32_t K, int64_t budget, int64_t cost_cap, int64_t* d_batch,
                               int32_t* d_best_k, int64_t* d_best_batch, int32_t* d_status, void* d_work,
                               size_t work_bytes, void* stream);

/* ---- execution plans ---------------------------------------------------
 * Algorithm 1 (Section 4.9): the program that carries out a schedule (S, R).
 * R is scanned row by row. In stage t, node k is computed into a new virtual
 * register when R[t][k] = 1 ("%r = compute v_k"; registers are numbered
 * 0, 1, ... in compute order). Then every i in Deps[k] u {k}, ascending, is
 * deallocated when FREE(t,i,k) = R[t][k] (1 - S[t+1][i]) prod over users
 * j > k of i of (1 - R[t][j]) holds (eq. collectable, S[n] = 0): each value
 * that is not kept goes right after its last computed use. A checkpoint with
 * no computed user in the stage that is not kept gets no FREE term. It is
 * deallocated at the end of the stage, where the U recurrence of Section 4.4
 * stops counting it. With CKM_PLAN_EARLY_FREE it is deallocated at the start
 * of the stage instead, the code motion Section 4.9 describes. Without that
 * flag, the memory after each compute equals U_{t,k} of the recurrence.
 *
 * S, R: n bit rows each, ceil(n/64) uint64 words per row, least significant
 * bit first (the layout of best_S / best_R). Entries of S with i >= t and of
 * R with i > t are ignored. (S, R) must satisfy R[t][t] = 1 (constraint 4a),
 * (1b), (1c), and S[t][i] R[t][i] = 0 (Algorithm 2's output does). Otherwise
 * the status is CKM_E_INVALID_ARG.
 * P: capacity statements (op, node, reg, stage). mem (may be NULL): capacity
 * int64 entries, the bytes in use after each statement, M_in + 2 M_param
 * included. count receives the plan's length, which is at most
 * CKM_PLAN_MAX_STMTS(n). With P NULL only the count is computed. If P is
 * given and capacity < count, the result is CKM_E_INVALID_ARG and nothing is
 * written to P. The synchronous form takes host arrays. The asynchronous
 * form takes device arrays, a work buffer from ckm_workspace_size(g, K) for
 * any K >= 1, and a stream. It writes the count and the status to d_count
 * and d_status (the latter may be NULL). */
typedef struct ckm_stmt {
  int32_t op;    /* CKM_OP_COMPUTE or CKM_OP_DEALLOCATE */
  int32_t node;  /* v_k computed, or the node whose value is deallocated */
  int32_t reg;   /* virtual register defined or released */
  int32_t stage; /* t */
} ckm_stmt;
enum { CKM_OP_COMPUTE = 0, CKM_OP_DEALLOCATE = 1 };
enum { CKM_PLAN_EARLY_FREE = 1u };
#define CKM_PLAN_MAX_STMTS(n) ((int64_t)(n) * ((int64_t)(n) + 1))

ckm_status ckm_plan(const ckm_graph* g, const uint64_t* S, const uint64_t* R, uint32_t flags, ckm_stmt* P,
                    int64_t capacity, int64_t* count, int64_t* mem);
ckm_status ckm_plan_async(const ckm_graph* g, const uint64_t* d_S, const uint64_t* d_R, uint32_t flags,
                          ckm_stmt* d_P, int64_t capacity, int64_t* d_count, int64_t* d_mem, int32_t* d_status,
                          void* d_work, size_t work_bytes, void* stream);

/* ---- no allocation -----------------------------------------------------
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.
 * ckm_round_eval_noalloc is ckm_round_eval_async (same arguments, same
 * results) with the caller's work buffer replaced by a static work area of
 * CKM_NOALLOC_SCRATCH_BYTES on each device, held from the library's first
 * use of the device until the process ends; its address is resolved when a
 * graph is created on the device. The call allocates nothing (no hipMalloc,
 * hipFree or other allocating routine) and only enqueues work on `stream`.
 * A problem whose smallest work buffer (ckm_workspace_size_min) exceeds the
 * area gives CKM_E_UNSUPPORTED; the row arrays are used when the full work
 * buffer (ckm_workspace_size) fits in it. Every call on one device shares
 * that device's area and the area keeps the last call's contents: calls
 * that may overlap on one device (other streams, other threads) race, and
 * the caller must serialize them. */
#define CKM_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)
ckm_status ckm_round_eval_noalloc(const ckm_graph* g, const double* d_s_frac, int64_t ld, int32_t K,
                                  uint64_t seed, int64_t budget, uint32_t flags, int64_t* d_peak,
                                  int64_t* d_cost, uint8_t* d_feasible, int32_t* d_best_k,
                                  uint64_t* d_best_S, uint64_t* d_best_R, int32_t* d_status, void* stream);

/* Thread-local text describing the calling thread's last non-OK status. */
const char* ckm_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
