/*
 * ckm_ref.c -- CPU oracle (test infrastructure only; see ckm_ref.h).
 *
 * Plain C99, single thread, no blocking, fusion or reordering beyond what the
 * definitions state. Each function names the passage of the paper it follows.
 */
#include "ckm_ref.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon et al., "Parallel random numbers: as easy as 1, 2,
 * 3", SC'11). Round: two 32x32->64 products of counter words 0 and 2 with
 * the multipliers; the new counter is (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1,
 * lo0); the key is advanced by the Weyl constants between rounds. */
#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void ckm_ref_philox4x32_10(const uint32_t key[2], const uint32_t ctr[4], uint32_t out[4]) {
  uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  int r;
  for (r = 0; r < 10; ++r) {
    uint64_t p0, p1;
    uint32_t n0, n1, n2, n3;
    if (r > 0) {
      k0 += PHILOX_W0;
      k1 += PHILOX_W1;
    }
    p0 = (uint64_t)PHILOX_M0 * (uint64_t)c0;
    p1 = (uint64_t)PHILOX_M1 * (uint64_t)c2;
    n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
    n1 = (uint32_t)p1;
    n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    n3 = (uint32_t)p0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

uint32_t ckm_ref_draw(uint64_t seed, uint32_t k, uint32_t t, uint32_t i) {
  uint32_t key[2], ctr[4], x[4];
  uint32_t j = i % 8u;
  key[0] = (uint32_t)(seed & 0xFFFFFFFFu);
  key[1] = (uint32_t)(seed >> 32);
  ctr[0] = i / 8u;
  ctr[1] = t;
  ctr[2] = k;
  ctr[3] = 0u;
  ckm_ref_philox4x32_10(key, ctr, x);
  return (x[j / 2u] >> (16u * (j % 2u))) & 0xFFFFu;
}

/* ------------------------------------------------------------------------ */
/* Section 4.1: a DAG whose nodes are numbered topologically, with per-node
 * output size M_v and compute cost C_v. */
int ckm_ref_validate_graph(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                           const int64_t* cost, const int64_t* size,
                           int64_t m_input, int64_t m_param) {
  int32_t j, a, b;
  int64_t total_m, total_c;
  if (n < 1 || !dep_ptr || !cost || !size) return CKM_REF_E_INVALID_ARG;
  if (dep_ptr[0] != 0) return CKM_REF_E_GRAPH;
  for (j = 0; j < n; ++j)
    if (dep_ptr[j + 1] < dep_ptr[j]) return CKM_REF_E_GRAPH;
  if (dep_ptr[n] > 0 && !dep_idx) return CKM_REF_E_INVALID_ARG;
  for (j = 0; j < n; ++j) {
    for (a = dep_ptr[j]; a < dep_ptr[j + 1]; ++a) {
      int32_t i = dep_idx[a];
      if (i < 0 || i >= j) return CKM_REF_E_GRAPH;            /* not topological */
      for (b = dep_ptr[j]; b < a; ++b)
        if (dep_idx[b] == i) return CKM_REF_E_GRAPH;          /* duplicate edge */
    }
  }
  if (m_input < 0 || m_param < 0) return CKM_REF_E_INVALID_ARG;
  for (j = 0; j < n; ++j)
    if (cost[j] < 0 || size[j] < 0) return CKM_REF_E_INVALID_ARG;
  /* M_in + 2 M_param + sum M must fit in int64 */
  total_m = m_input;
  if (m_param > INT64_MAX - total_m) return CKM_REF_E_OVERFLOW;
  total_m += m_param;
  if (m_param > INT64_MAX - total_m) return CKM_REF_E_OVERFLOW;
  total_m += m_param;
  for (j = 0; j < n; ++j) {
    if (size[j] > INT64_MAX - total_m) return CKM_REF_E_OVERFLOW;
    total_m += size[j];
  }
  /* n * sum C must fit in int64 (every stage may compute every node) */
  total_c = 0;
  for (j = 0; j < n; ++j) {
    if (cost[j] > INT64_MAX - total_c) return CKM_REF_E_OVERFLOW;
    total_c += cost[j];
  }
  if (total_c > 0 && (int64_t)n > INT64_MAX / total_c) return CKM_REF_E_OVERFLOW;
  return CKM_REF_OK;
}

/* ------------------------------------------------------------------------ */
/* Section 5.1: randomized rounding takes x_int = 1 with probability x*. The
 * probability is quantized to 16 bits: q = floor(x* * 2^16), so that
 * Pr[u < q] = q / 2^16 lies in (x* - 2^-16, x*]. */
int ckm_ref_quantize(int32_t n, const double* s_frac, int64_t ld, uint32_t* q) {
  int32_t t, i;
  for (t = 0; t < n; ++t) {
    for (i = 0; i < n; ++i) {
      uint32_t v = 0;
      if (i < t) {
        double x = s_frac[(int64_t)t * ld + i];
        if (isnan(x)) return CKM_REF_E_INVALID_ARG;
        if (x < 0.0) x = 0.0;
        if (x > 1.0) x = 1.0;
        v = (uint32_t)floor(x * 65536.0);
      }
      q[(int64_t)t * n + i] = v;
    }
  }
  return CKM_REF_OK;
}

void ckm_ref_round_random(int32_t n, const uint32_t* q, uint64_t seed, uint32_t k, uint8_t* S) {
  int32_t t, i;
  for (t = 0; t < n; ++t)
    for (i = 0; i < n; ++i) {
      uint8_t s = 0;
      if (i < t) s = ckm_ref_draw(seed, k, (uint32_t)t, (uint32_t)i) < q[(int64_t)t * n + i];
      S[(int64_t)t * n + i] = s;
    }
}

/* The deterministic rounding of Algorithm 2: S_int = 1[S* > 0.5]. */
void ckm_ref_round_det(int32_t n, const double* s_frac, int64_t ld, uint8_t* S) {
  int32_t t, i;
  for (t = 0; t < n; ++t)
    for (i = 0; i < n; ++i)
      S[(int64_t)t * n + i] = (i < t) && (s_frac[(int64_t)t * ld + i] > 0.5);
}

/* Deterministic rounding at a chosen threshold p (Section 5.1 rounds
 * x_int = 1[x* >= p]; Algorithm 2 takes p = 0.5 with a strict comparison, the
 * form used here): S[t][i] = [clamp(S*[t][i], 0, 1) > p] for i < t, compared
 * in double. A NaN entry of the strict lower triangle, or a NaN p, is an
 * argument error. */
int ckm_ref_round_threshold(int32_t n, const double* s_frac, int64_t ld, double p, uint8_t* S) {
  int32_t t, i;
  if (isnan(p)) return CKM_REF_E_INVALID_ARG;
  for (t = 0; t < n; ++t)
    for (i = 0; i < n; ++i) {
      uint8_t v = 0;
      if (i < t) {
        double x = s_frac[(int64_t)t * ld + i];
        if (isnan(x)) return CKM_REF_E_INVALID_ARG;
        if (x < 0.0) x = 0.0;
        if (x > 1.0) x = 1.0;
        v = x > p;
      }
      S[(int64_t)t * n + i] = v;
    }
  return CKM_REF_OK;
}

/* ------------------------------------------------------------------------ */
/* The recomputation matrix of two-phase rounding (Section 5.2), from the
 * constraints it has to satisfy rather than from the repair loops of the
 * printed listing. For stage t, R_t must contain node t (constraint 4a),
 * every value kept for stage t+1 that stage t does not already hold
 * (constraint 1c: S[t+1][i] <= R[t][i] + S[t][i]), and every dependency of a
 * computed node that stage t does not hold (constraint 1b: R[t][j] <=
 * R[t][i] + S[t][i] for each edge (i, j)). Section 5.2 takes the smallest such
 * R_t, and the conditions are monotone, so R_t is the set reached from those
 * seeds by walking dependency edges backwards, never into a value of S_t:
 * a least fixed point, found here by a plain worklist search. */
void ckm_ref_solve_R(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                     const uint8_t* S, uint8_t* R) {
  int32_t* stack = (int32_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
  int32_t t, i, a, top;
  memset(R, 0, (size_t)n * (size_t)n);
  for (t = 0; t < n; ++t) {
    const uint8_t* St = S + (int64_t)t * n;
    const uint8_t* Snext = (t + 1 < n) ? S + (int64_t)(t + 1) * n : NULL;  /* S[n] = 0 */
    uint8_t* Rt = R + (int64_t)t * n;
    top = 0;
    /* seeds: node t (4a), values kept into t+1 but not held in t (1c) */
    Rt[t] = 1;
    stack[top++] = t;
    for (i = 0; i < t; ++i)
      if (Snext && Snext[i] && !St[i] && !Rt[i]) {
        Rt[i] = 1;
        stack[top++] = i;
      }
    /* closure under (1b): an operand of a computed node that is not held */
    while (top > 0) {
      int32_t j = stack[--top];
      for (a = dep_ptr[j]; a < dep_ptr[j + 1]; ++a) {
        i = dep_idx[a];
        if (!St[i] && !Rt[i]) {
          Rt[i] = 1;
          stack[top++] = i;
        }
      }
    }
  }
  free(stack);
}

/* ------------------------------------------------------------------------ */
/* Section 4.4. Memory in use at the start of stage t (eq. U_init):
 *   U_{t,0} = M_in + 2 M_param + sum_i M_i S[t][i];
 * after computing v_k (eq. mem_recurrence): U_{t,k} = U_{t,k-1} - freed(k-1)
 *   + R[t][k] M_k, where freed(k) = sum over i in Deps[k] u {k} of
 *   M_i FREE(t,i,k) (eq. GC) and
 *   FREE(t,i,k) = R[t][k] (1 - S[t+1][i]) prod_{j in Users[i], j > k} (1 - R[t][j])
 *   (eq. collectable). The i = k term is kept (it is only dropped from the
 *   ILP as implied by optimality, Section 4.8).
 * The objective of Section 4.3 gives the cost: sum_t sum_i C_i R[t][i]. */
void ckm_ref_simulate(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                      const int64_t* cost, const int64_t* size, int64_t m_input, int64_t m_param,
                      const uint8_t* S, const uint8_t* R, int64_t* peak, int64_t* total_cost,
                      int64_t* stage_peak, int32_t* max_frees, int64_t* U_end) {
  int32_t t, i, k, a, b, j;
  int32_t E = dep_ptr[n];
  int32_t* user_ptr = (int32_t*)calloc((size_t)n + 1, sizeof(int32_t));
  int32_t* user_idx = (int32_t*)malloc((size_t)(E > 0 ? E : 1) * sizeof(int32_t));
  int32_t* fill = (int32_t*)calloc((size_t)n, sizeof(int32_t));
  int32_t* free_count = (int32_t*)calloc((size_t)n, sizeof(int32_t));
  int64_t best = INT64_MIN, csum = 0;
  int32_t worst_frees = 0;

  /* Users[i] = { j : (v_i, v_j) in E } (transpose of Deps) */
  for (j = 0; j < n; ++j)
    for (a = dep_ptr[j]; a < dep_ptr[j + 1]; ++a) user_ptr[dep_idx[a] + 1]++;
  for (i = 0; i < n; ++i) user_ptr[i + 1] += user_ptr[i];
  for (j = 0; j < n; ++j)
    for (a = dep_ptr[j]; a < dep_ptr[j + 1]; ++a) {
      i = dep_idx[a];
      user_idx[user_ptr[i] + fill[i]++] = j;
    }

  for (t = 0; t < n; ++t) {
    const uint8_t* St = S + (int64_t)t * n;
    const uint8_t* Rt = R + (int64_t)t * n;
    const uint8_t* Snext = (t + 1 < n) ? S + (int64_t)(t + 1) * n : NULL;  /* S[n] = 0 */
    int64_t U = m_input + 2 * m_param;
    int64_t speak = INT64_MIN;
    for (i = 0; i < n; ++i) U += size[i] * (int64_t)St[i];
    memset(free_count, 0, (size_t)n * sizeof(int32_t));
    for (k = 0; k < n; ++k) {
      int64_t freed = 0;
      int32_t m;
      U += (int64_t)Rt[k] * size[k];
      if (U > speak) speak = U;
      /* i ranges over Deps[k] u {k}; m = 0 .. deg(k)-1 are the deps, m = deg(k) is k */
      for (m = 0; m <= dep_ptr[k + 1] - dep_ptr[k]; ++m) {
        int64_t FREE;
        i = (m < dep_ptr[k + 1] - dep_ptr[k]) ? dep_idx[dep_ptr[k] + m] : k;
        FREE = (int64_t)Rt[k] * (1 - (int64_t)(Snext ? Snext[i] : 0));
        for (b = user_ptr[i]; b < user_ptr[i + 1]; ++b) {
          j = user_idx[b];
          if (j > k) FREE *= (1 - (int64_t)Rt[j]);
        }
        freed += size[i] * FREE;
        free_count[i] += (int32_t)FREE;
      }
      U -= freed;
    }
    for (i = 0; i < n; ++i) {
      csum += cost[i] * (int64_t)Rt[i];
      if (free_count[i] > worst_frees) worst_frees = free_count[i];
    }
    if (stage_peak) stage_peak[t] = speak;
    if (U_end) U_end[t] = U;
    if (speak > best) best = speak;
  }
  *peak = best;
  *total_cost = csum;
  if (max_frees) *max_frees = worst_frees;
  free(user_ptr);
  free(user_idx);
  free(fill);
  free(free_count);
}

/* ------------------------------------------------------------------------ */
int ckm_ref_eval_candidate(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                           const int64_t* cost, const int64_t* size, int64_t m_input,
                           int64_t m_param, const double* s_frac, int64_t ld, const uint32_t* q,
                           uint64_t seed, uint32_t k, uint32_t flags, int64_t* peak,
                           int64_t* total_cost, uint8_t* S_out, uint8_t* R_out) {
  size_t nn = (size_t)n * (size_t)n;
  uint8_t* S = S_out ? S_out : (uint8_t*)malloc(nn);
  uint8_t* R = R_out ? R_out : (uint8_t*)malloc(nn);
  if (!S || !R) return CKM_REF_E_INVALID_ARG;
  if (k == 0 && (flags & CKM_REF_F_DET0))
    ckm_ref_round_det(n, s_frac, ld, S);
  else
    ckm_ref_round_random(n, q, seed, k, S);
  ckm_ref_solve_R(n, dep_ptr, dep_idx, S, R);
  ckm_ref_simulate(n, dep_ptr, dep_idx, cost, size, m_input, m_param, S, R, peak, total_cost,
                   NULL, NULL, NULL);
  if (!S_out) free(S);
  if (!R_out) free(R);
  return CKM_REF_OK;
}

static void pack_rows(int32_t n, const uint8_t* X, uint64_t* out) {
  int32_t W = (n + 63) / 64, t, i;
  memset(out, 0, (size_t)n * (size_t)W * sizeof(uint64_t));
  for (t = 0; t < n; ++t)
    for (i = 0; i < n; ++i)
      if (X[(int64_t)t * n + i]) out[(int64_t)t * W + i / 64] |= (uint64_t)1 << (i % 64);
}

int ckm_ref_round_eval(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                       const int64_t* cost, const int64_t* size, int64_t m_input, int64_t m_param,
                       const double* s_frac, int64_t ld, int32_t K, uint64_t seed, int64_t budget,
                       uint32_t flags, int64_t* peak, int64_t* total_cost, uint8_t* feasible,
                       int32_t* best_k, uint64_t* best_S, uint64_t* best_R) {
  int st;
  int32_t k, bk = -1;
  uint32_t* q;
  size_t nn = (size_t)n * (size_t)n;
  if (K < 1 || !s_frac || ld < n || budget < 0 || !peak || !total_cost || !feasible || !best_k)
    return CKM_REF_E_INVALID_ARG;
  st = ckm_ref_validate_graph(n, dep_ptr, dep_idx, cost, size, m_input, m_param);
  if (st != CKM_REF_OK) return st;
  q = (uint32_t*)malloc(nn * sizeof(uint32_t));
  st = ckm_ref_quantize(n, s_frac, ld, q);
  if (st != CKM_REF_OK) { free(q); return st; }
  for (k = 0; k < K; ++k) {
    ckm_ref_eval_candidate(n, dep_ptr, dep_idx, cost, size, m_input, m_param, s_frac, ld, q, seed,
                           (uint32_t)k, flags, &peak[k], &total_cost[k], NULL, NULL);
    feasible[k] = peak[k] <= budget;
    /* best = lexicographic minimum of (cost, peak, k) over feasible k */
    if (feasible[k] && (bk < 0 || total_cost[k] < total_cost[bk] ||
                        (total_cost[k] == total_cost[bk] && peak[k] < peak[bk])))
      bk = k;
  }
  *best_k = bk;
  if (best_S || best_R) {
    int32_t W = (n + 63) / 64;
    if (bk >= 0) {
      uint8_t* S = (uint8_t*)malloc(nn);
      uint8_t* R = (uint8_t*)malloc(nn);
      int64_t p, c;
      ckm_ref_eval_candidate(n, dep_ptr, dep_idx, cost, size, m_input, m_param, s_frac, ld, q,
                             seed, (uint32_t)bk, flags, &p, &c, S, R);
      if (best_S) pack_rows(n, S, best_S);
      if (best_R) pack_rows(n, R, best_R);
      free(S);
      free(R);
    } else {
      if (best_S) memset(best_S, 0, (size_t)n * (size_t)W * sizeof(uint64_t));
      if (best_R) memset(best_R, 0, (size_t)n * (size_t)W * sizeof(uint64_t));
    }
  }
  free(q);
  return CKM_REF_OK;
}

/* ------------------------------------------------------------------------ */
/* Conditions the plan generator needs of (S, R), strict lower S and lower R
 * (entries of S with i >= t and of R with i > t are not read):
 *   R[t][t] = 1 (constraint 4a); no value both kept and recomputed in one
 *   stage (R[t][i] S[t][i] = 0, which Algorithm 2's output satisfies);
 *   (1b) R[t][j] <= R[t][i] + S[t][i] for every edge (i, j);
 *   (1c) S[t+1][i] <= R[t][i] + S[t][i].
 * Returns CKM_REF_OK or CKM_REF_E_INVALID_ARG. */
int ckm_ref_check_schedule(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                           const uint8_t* S, const uint8_t* R) {
  int32_t t, i, j, a;
#define SB(t, i) ((i) < (t) ? S[(int64_t)(t) * n + (i)] : 0)
#define RB(t, i) ((i) <= (t) ? R[(int64_t)(t) * n + (i)] : 0)
  for (t = 0; t < n; ++t) {
    if (!RB(t, t)) return CKM_REF_E_INVALID_ARG;
    for (i = 0; i < t; ++i)
      if (SB(t, i) && RB(t, i)) return CKM_REF_E_INVALID_ARG;
    for (j = 0; j <= t; ++j)
      if (RB(t, j))
        for (a = dep_ptr[j]; a < dep_ptr[j + 1]; ++a) {
          i = dep_idx[a];
          if (!RB(t, i) && !SB(t, i)) return CKM_REF_E_INVALID_ARG;
        }
    if (t + 1 < n)
      for (i = 0; i <= t; ++i)
        if (SB(t + 1, i) && !RB(t, i) && !SB(t, i)) return CKM_REF_E_INVALID_ARG;
  }
#undef SB
#undef RB
  return CKM_REF_OK;
}

/* The execution plan of Section 4.9 for a schedule (S, R), built from the
 * memory model of Section 4.4 rather than by retracing the printed listing.
 * Within stage t the plan computes, in increasing node order, every node
 * with R[t][k] = 1, each into a fresh virtual register (registers numbered
 * in compute order). A value i is released at the node k for which
 * FREE(t,i,k) = 1 (eq. collectable: k computed, i in Deps[k] u {k}, i not
 * kept into stage t+1, and no user of i after k computed in the stage);
 * Theorem 4.1 makes that k unique. The release follows the compute of k, and
 * releases at one k go in increasing order of the value (so k itself, the
 * largest, comes last). A value held at the start of the stage that no
 * computed node uses and that is not kept has no FREE term; it is released
 * at the end of the stage, where the U recurrence stops counting it, or with
 * early != 0 at the start (the code motion Section 4.9 describes).
 * Statement s is stmts[4s .. 4s+3] = (op, node, register, stage), op 0 =
 * compute, 1 = deallocate. mem[s] (may be NULL) = M_in + 2 M_param plus the
 * sizes of the registers live after statement s. At most `capacity`
 * statements are written; *count receives the plan's length. Returns
 * CKM_REF_E_INVALID_ARG when (S, R) fails ckm_ref_check_schedule. */
int ckm_ref_plan(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx, const int64_t* size,
                 int64_t m_input, int64_t m_param, const uint8_t* S, const uint8_t* R, int early,
                 int32_t* stmts, int64_t* mem, int64_t capacity, int64_t* count) {
  int32_t t, k, i, j, a, b;
  int64_t s = 0, r = 0, live_bytes = 0;
  int32_t* reg;       /* register holding value i, -1 if none */
  int32_t* free_at;   /* per stage: the k with FREE(t,i,k) = 1, or -1 */
  int32_t* user_ptr;
  int32_t* user_idx;
  int32_t* fill;
  int32_t E = dep_ptr[n];
  int st = ckm_ref_check_schedule(n, dep_ptr, dep_idx, S, R);
  if (st != CKM_REF_OK) return st;
  reg = (int32_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
  free_at = (int32_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
  user_ptr = (int32_t*)calloc((size_t)n + 1, sizeof(int32_t));
  user_idx = (int32_t*)malloc((size_t)(E > 0 ? E : 1) * sizeof(int32_t));
  fill = (int32_t*)calloc((size_t)n, sizeof(int32_t));
  for (i = 0; i < n; ++i) reg[i] = -1;
  /* Users[i] = { j : (v_i, v_j) in E } (transpose of Deps) */
  for (j = 0; j < n; ++j)
    for (a = dep_ptr[j]; a < dep_ptr[j + 1]; ++a) user_ptr[dep_idx[a] + 1]++;
  for (i = 0; i < n; ++i) user_ptr[i + 1] += user_ptr[i];
  for (j = 0; j < n; ++j)
    for (a = dep_ptr[j]; a < dep_ptr[j + 1]; ++a) {
      i = dep_idx[a];
      user_idx[user_ptr[i] + fill[i]++] = j;
    }

#define EMIT(op_, node_, reg_)                                                  \
  do {                                                                          \
    live_bytes += (op_) == 0 ? size[node_] : -size[node_];                      \
    if (s < capacity) {                                                         \
      stmts[4 * s] = (op_);                                                     \
      stmts[4 * s + 1] = (node_);                                               \
      stmts[4 * s + 2] = (int32_t)(reg_);                                       \
      stmts[4 * s + 3] = t;                                                     \
      if (mem) mem[s] = m_input + 2 * m_param + live_bytes;                     \
    }                                                                           \
    ++s;                                                                        \
  } while (0)
#define KEPT(i_) (t + 1 < n && (i_) < t + 1 && S[(int64_t)(t + 1) * n + (i_)])

  for (t = 0; t < n; ++t) {
    const uint8_t* St = S + (int64_t)t * n;
    const uint8_t* Rt = R + (int64_t)t * n;
    /* free point of each value: eq. collectable evaluated for every pair
     * (i, k) with i in Deps[k] u {k} */
    for (i = 0; i < n; ++i) free_at[i] = -1;
    for (k = 0; k <= t; ++k) {
      if (!Rt[k]) continue;
      for (a = dep_ptr[k]; a <= dep_ptr[k + 1]; ++a) {
        int later = 0;
        i = (a < dep_ptr[k + 1]) ? dep_idx[a] : k;
        if (KEPT(i)) continue;
        for (b = user_ptr[i]; b < user_ptr[i + 1]; ++b) {
          j = user_idx[b];
          if (j > k && j <= t && Rt[j]) later = 1;
        }
        if (!later) free_at[i] = k;
      }
    }
    /* unused checkpoints not kept into t+1: released at the start (early) */
    if (early)
      for (i = 0; i < t; ++i)
        if (St[i] && free_at[i] < 0 && !KEPT(i)) EMIT(1, i, reg[i]);
    for (k = 0; k <= t; ++k) {
      if (!Rt[k]) continue;
      reg[k] = (int32_t)r;
      EMIT(0, k, r);
      ++r;
      for (i = 0; i <= k; ++i)
        if (free_at[i] == k) EMIT(1, i, reg[i]);
    }
    /* ... or at the end of the stage */
    if (!early)
      for (i = 0; i < t; ++i)
        if (St[i] && free_at[i] < 0 && !KEPT(i)) EMIT(1, i, reg[i]);
  }
#undef KEPT
#undef EMIT
  *count = s;
  free(reg);
  free(free_at);
  free(user_ptr);
  free(user_idx);
  free(fill);
  return CKM_REF_OK;
}

/* ------------------------------------------------------------------------ */
/* Largest batch multiplier of one schedule (the maximum-batch experiment of
 * the evaluation): node sizes become B * M_i (M_input and M_param stay), and
 * B is the largest integer with peak memory <= budget, subject to the cost
 * cap of eq. (cost_constr) (costs do not scale with B). Found by search over
 * the simulator: doubling, then bisection. 0 when B = 1 already fails or the
 * cost exceeds the cap; limit when B = limit still fits. */
int64_t ckm_ref_max_batch(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx, const int64_t* cost,
                          const int64_t* size, int64_t m_input, int64_t m_param, const uint8_t* S,
                          const uint8_t* R, int64_t budget, int64_t cost_cap, int64_t limit) {
  int64_t* scaled = (int64_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
  int64_t lo = 0, hi, peak, c;
  int32_t i;
#define FITS(B_, out_)                                                                     \
  do {                                                                                     \
    for (i = 0; i < n; ++i) scaled[i] = (B_) * size[i];                                    \
    ckm_ref_simulate(n, dep_ptr, dep_idx, cost, scaled, m_input, m_param, S, R, &peak, &c, \
                     NULL, NULL, NULL);                                                    \
    (out_) = peak <= budget;                                                               \
  } while (0)
  {
    int ok;
    FITS((int64_t)1, ok);
    if (!ok || c > cost_cap) {
      free(scaled);
      return 0;
    }
  }
  lo = 1;
  hi = 2;
  for (;;) {   /* doubling: lo fits, find hi that does not (or reach the limit) */
    int ok;
    if (hi >= limit) {
      FITS(limit, ok);
      if (ok) {
        free(scaled);
        return limit;
      }
      hi = limit;
      break;
    }
    FITS(hi, ok);
    if (!ok) break;
    lo = hi;
    hi *= 2;
  }
  while (hi - lo > 1) {   /* lo fits, hi does not */
    int64_t mid = lo + (hi - lo) / 2;
    int ok;
    FITS(mid, ok);
    if (ok) lo = mid;
    else hi = mid;
  }
#undef FITS
  free(scaled);
  return lo;
}
