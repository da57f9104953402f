// Execution plan of one schedule (S, R) on the GPU (Section 4.9, Algorithm 1).
//
// Algorithm 1 scans R row by row: in stage t, node k is computed into a new
// virtual register when R[t][k] = 1, and then every i in Deps[k] u {k} with
// FREE(t,i,k) = 1 is deallocated. Each stage's statements depend only on
// rows t and t+1, so stages are independent once two prefix sums are known:
// the first statement of each stage (statement counts) and the first
// register of each stage (compute counts, since registers are numbered in
// compute order). Three launches:
//   count: one wave per stage: statement and compute counts, and the checks
//          the plan relies on ((4a), (1b), (1c), no value both kept and
//          recomputed);
//   scan:  one block: the two prefix sums, the total, the status;
//   emit:  one wave per stage writes its statements at their final
//          positions, with the memory in use after each.
//
// FREE(t,i,k) = R[t][k] (1 - S[t+1][i]) prod_{j in Users[i], j > k} (1 - R[t][j])
// is 1 for exactly one k when value i is live in stage t and not kept: its
// last computed user in the stage, or i itself when no user is computed and
// i is computed (Theorem 4.1). A checkpoint with no computed user that is
// not kept gets no FREE term; it is deallocated at the end of the stage (the
// U recurrence counts it to there) or, with CKM_PLAN_EARLY_FREE, at the
// start (the code motion of Section 4.9). So a stage has
// popcount(R_t) + popcount((S_t | R_t) & ~S_{t+1}) statements.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "ckm_internal.h"

namespace ckm {
namespace {

constexpr int kPlanWave = 64;
constexpr int kFreeNone = -1;    // not freed in this stage (dead, or kept)
constexpr int kFreeUnused = -2;  // unused checkpoint, not kept: stage start or end

__device__ __forceinline__ uint32_t bit_of(uint32_t word, int i) { return (word >> (i & 31)) & 1u; }

// Word w of S row t restricted to i < t, and of R row t restricted to i <= t.
__device__ __forceinline__ uint32_t s_word(const uint32_t* S, int rw, int t, int w) {
  const int lo = 32 * w;
  if (lo >= t) return 0u;
  const uint32_t v = S[(size_t)t * rw + w];
  return (t - lo >= 32) ? v : (v & ((1u << (t - lo)) - 1u));
}
__device__ __forceinline__ uint32_t r_word(const uint32_t* R, int rw, int t, int w) {
  const int lo = 32 * w;
  if (lo > t) return 0u;
  const uint32_t v = R[(size_t)t * rw + w];
  return (t - lo >= 31) ? v : (v & ((2u << (t - lo)) - 1u));
}

__device__ __forceinline__ int64_t wave_sum_i64(int64_t x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}
__device__ __forceinline__ double wave_sum_f64(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}
// Inclusive prefix sums over the lanes of the wave.
__device__ __forceinline__ int64_t wave_scan_i64(int64_t x, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  return x;
}
__device__ __forceinline__ double wave_scan_f64(double x, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  return x;
}

// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kPlanWave) ckm_plan_count_kernel(int32_t n, int32_t rw,
                                                                   const uint32_t* __restrict__ S,
                                                                   const uint32_t* __restrict__ R,
                                                                   const int32_t* __restrict__ dep_ptr,
                                                                   const int32_t* __restrict__ dep_idx,
                                                                   int64_t* __restrict__ cnt,
                                                                   int64_t* __restrict__ comp,
                                                                   int32_t* __restrict__ err) {
  const int t = blockIdx.x;
  const int lane = threadIdx.x;
  const int nwt = (t >> 5) + 1;
  int64_t c = 0, f = 0;
  uint32_t bad = 0;
  for (int w = lane; w < nwt; w += kPlanWave) {
    const uint32_t s = s_word(S, rw, t, w);
    const uint32_t r = r_word(R, rw, t, w);
    const uint32_t sn = (t + 1 < n) ? s_word(S, rw, t + 1, w) : 0u;
    c += __popc(r);
    f += __popc((s | r) & ~sn);
    bad |= (s & r) != 0u;              // kept and recomputed
    bad |= (sn & ~(s | r)) != 0u;      // (1c)
    if (w == (t >> 5)) bad |= bit_of(r, t) ^ 1u;   // (4a)
    // (1b): every dep of a computed node is resident
    uint32_t m = r;
    while (m) {
      const int k = 32 * w + __ffs(m) - 1;
      m &= m - 1u;
      for (int e = dep_ptr[k]; e < dep_ptr[k + 1]; ++e) {
        const int i = dep_idx[e];
        const uint32_t have = s_word(S, rw, t, i >> 5) | r_word(R, rw, t, i >> 5);
        bad |= bit_of(have, i) ^ 1u;
      }
    }
  }
  c = wave_sum_i64(c);
  f = wave_sum_i64(f);
  const uint64_t any_bad = __ballot(bad != 0u);
  if (lane == 0) {
    cnt[t] = c + f;
    comp[t] = c;
    err[t] = any_bad ? 1 : 0;
  }
}

// One block: exclusive prefix sums of the statement and compute counts, the
// total, and the status. go = 1 when statements are to be written.
constexpr int kScanThreads = 1024;
__global__ void __launch_bounds__(kScanThreads) ckm_plan_scan_kernel(
    int32_t n, const int64_t* __restrict__ cnt, const int64_t* __restrict__ comp,
    const int32_t* __restrict__ err, int64_t* __restrict__ off, int64_t* __restrict__ rbase,
    int64_t capacity, int32_t want_stmts, int64_t* __restrict__ d_count, int32_t* __restrict__ d_status,
    int32_t* __restrict__ go) {
  __shared__ int64_t sc[kScanThreads], sr[kScanThreads];
  __shared__ int any_err;
  const int tid = threadIdx.x;
  const int per = (n + kScanThreads - 1) / kScanThreads;
  const int a = tid * per, b = min(n, a + per);
  if (tid == 0) any_err = 0;
  __syncthreads();
  int64_t c = 0, r = 0;
  int e = 0;
  for (int t = a; t < b; ++t) {
    c += cnt[t];
    r += comp[t];
    e |= err[t];
  }
  if (e) atomicOr(&any_err, 1);
  sc[tid] = c;
  sr[tid] = r;
  __syncthreads();
  for (int o = 1; o < kScanThreads; o <<= 1) {
    const int64_t xc = tid >= o ? sc[tid - o] : 0;
    const int64_t xr = tid >= o ? sr[tid - o] : 0;
    __syncthreads();
    sc[tid] += xc;
    sr[tid] += xr;
    __syncthreads();
  }
  int64_t pc = sc[tid] - c, pr = sr[tid] - r;   // exclusive
  for (int t = a; t < b; ++t) {
    off[t] = pc;
    rbase[t] = pr;
    pc += cnt[t];
    pr += comp[t];
  }
  if (tid == kScanThreads - 1) {
    const int64_t total = sc[kScanThreads - 1];
    const bool fits = !want_stmts || total <= capacity;
    const int32_t st = any_err ? (int32_t)CKM_E_INVALID_ARG : (fits ? (int32_t)CKM_OK : (int32_t)CKM_E_INVALID_ARG);
    d_count[0] = total;
    if (d_status) d_status[0] = st;
    go[0] = (st == CKM_OK && want_stmts) ? 1 : 0;
  }
}

struct PlanArgs {
  int32_t n, rw;
  int32_t early;
  double base;                       // M_in + 2 M_param
  const uint32_t* S;
  const uint32_t* R;
  const int32_t* dep_ptr;
  const int32_t* dep_idx;
  const int32_t* user_ptr;
  const int32_t* user_idx;
  const double* M;
  const int64_t* off;
  const int64_t* rbase;
  const int32_t* go;
  int32_t* P;                        // [capacity][4]: op, node, register, stage
  int64_t* mem;                      // [capacity] or null
  int64_t capacity;
};

__device__ __forceinline__ void put_stmt(const PlanArgs& a, int64_t s, int op, int node, int64_t reg, int t,
                                         double mem_after) {
  // positions come from the count kernel's totals, which the scan checked
  // against the capacity; the guard keeps every store inside the buffers
  if (s < 0 || s >= a.capacity) return;
  int32_t* p = a.P + 4 * s;
  p[0] = op;
  p[1] = node;
  p[2] = (int32_t)reg;
  p[3] = t;
  if (a.mem) a.mem[s] = (int64_t)mem_after;
}

// Register of value i live in stage t: computed in this stage, or the
// register of the stage s < t that computed the checkpoint: the last stage
// s <= t with S[s][i] = 0 (constraint (1c) then has R[s][i] = 1).
__device__ int64_t reg_of(const PlanArgs& a, int t, int i, const uint32_t* rt_lds, const int32_t* wpre) {
  const int w = i >> 5;
  const uint32_t below = (1u << (i & 31)) - 1u;
  if (bit_of(rt_lds[w], i)) return (int64_t)wpre[w] + __popc(rt_lds[w] & below) + a.rbase[t];
  int s = t - 1;
  while (s > i && bit_of(s_word(a.S, a.rw, s, w), i)) --s;
  int64_t rank = 0;
  for (int v = 0; v < w; ++v) rank += __popc(r_word(a.R, a.rw, s, v));
  rank += __popc(r_word(a.R, a.rw, s, w) & below);
  return a.rbase[s] + rank;
}

// Stage t: one wave. LDS holds the stage's rows, the per-word compute counts
// of R_t and each node's free point.
__global__ void __launch_bounds__(kPlanWave) ckm_plan_emit_kernel(PlanArgs a) {
  __shared__ uint32_t st_l[kMaxNodesWords], rt_l[kMaxNodesWords], sn_l[kMaxNodesWords];
  __shared__ int32_t wpre[kMaxNodesWords];
  __shared__ int32_t fpt[CKM_MAX_NODES];
  const int t = blockIdx.x;
  const int lane = threadIdx.x;
  if (a.go[0] == 0) return;
  const int nwt = (t >> 5) + 1;
  for (int w = lane; w < nwt; w += kPlanWave) {
    st_l[w] = s_word(a.S, a.rw, t, w);
    rt_l[w] = r_word(a.R, a.rw, t, w);
    sn_l[w] = (t + 1 < a.n) ? s_word(a.S, a.rw, t + 1, w) : 0u;
  }
  __syncthreads();
  // computes in the words before w (nwt <= 128: two rounds of 64 lanes)
  {
    int64_t carry = 0;
    for (int w0 = 0; w0 < nwt; w0 += kPlanWave) {
      const int w = w0 + lane;
      const int64_t c = w < nwt ? __popc(rt_l[w]) : 0;
      const int64_t inc = wave_scan_i64(c, lane);
      if (w < nwt) wpre[w] = (int32_t)(carry + inc - c);
      carry += __shfl(inc, kPlanWave - 1);
    }
  }
  // free point of each node and the stage's starting memory
  double kept_bytes = 0.0;
  for (int i = lane; i <= t; i += kPlanWave) {
    const uint32_t si = bit_of(st_l[i >> 5], i), ri = bit_of(rt_l[i >> 5], i);
    int f = kFreeNone;
    if ((si | ri) && !bit_of(sn_l[i >> 5], i)) {
      f = ri ? i : kFreeUnused;
      for (int e = a.user_ptr[i + 1] - 1; e >= a.user_ptr[i]; --e) {
        const int j = a.user_idx[e];
        if (j <= t && bit_of(rt_l[j >> 5], j)) {
          f = j;
          break;
        }
      }
    }
    fpt[i] = f;
    if (si) kept_bytes += a.M[i];
  }
  __syncthreads();
  double u = a.base + wave_sum_f64(kept_bytes);   // U_{t,0}: exact integer
  int64_t pos = a.off[t];

  // unused checkpoints, ascending; at the start (early) or at the end
  auto unused_pass = [&]() {
    for (int i0 = 0; i0 <= t; i0 += kPlanWave) {
      const int i = i0 + lane;
      const bool fl = i <= t && fpt[i] == kFreeUnused;
      const uint64_t mask = __ballot(fl);
      if (!mask) continue;
      const int idx = __popcll(mask & ((1ull << lane) - 1ull));
      const double d = fl ? -a.M[i] : 0.0;
      const double incl = wave_scan_f64(d, lane);
      if (fl) put_stmt(a, pos + idx, 1, i, reg_of(a, t, i, rt_l, wpre), t, u + incl);
      pos += __popcll(mask);
      u += __shfl(incl, kPlanWave - 1);
    }
  };
  if (a.early) unused_pass();

  // the scan of Algorithm 1, 64 nodes at a time
  for (int k0 = 0; k0 <= t; k0 += kPlanWave) {
    const int k = k0 + lane;
    int64_t c = 0;
    double d = 0.0;
    const bool in = k <= t;
    const bool rk = in && bit_of(rt_l[k >> 5], k);
    if (in) {
      if (rk) {
        c = 1;
        d = a.M[k];
      }
      for (int e = a.dep_ptr[k]; e < a.dep_ptr[k + 1]; ++e) {
        const int i = a.dep_idx[e];
        if (fpt[i] == k) {
          ++c;
          d -= a.M[i];
        }
      }
      if (fpt[k] == k) {
        ++c;
        d -= a.M[k];
      }
    }
    const int64_t cinc = wave_scan_i64(c, lane);
    const double dinc = wave_scan_f64(d, lane);
    int64_t s = pos + cinc - c;
    double mu = u + dinc - d;      // memory before this node's statements
    if (c) {
      if (rk) {
        mu += a.M[k];
        const int64_t reg = a.rbase[t] + wpre[k >> 5] + __popc(rt_l[k >> 5] & ((1u << (k & 31)) - 1u));
        put_stmt(a, s++, 0, k, reg, t, mu);
      }
      for (int e = a.dep_ptr[k]; e < a.dep_ptr[k + 1]; ++e) {
        const int i = a.dep_idx[e];
        if (fpt[i] == k) {
          mu -= a.M[i];
          put_stmt(a, s++, 1, i, reg_of(a, t, i, rt_l, wpre), t, mu);
        }
      }
      if (fpt[k] == k) {
        mu -= a.M[k];
        put_stmt(a, s++, 1, k, reg_of(a, t, k, rt_l, wpre), t, mu);
      }
    }
    pos += __shfl(cinc, kPlanWave - 1);
    u += __shfl(dinc, kPlanWave - 1);
  }
  if (!a.early) unused_pass();
}

template <typename T>
T* at(char* work, size_t off) { return reinterpret_cast<T*>(work + off); }

}  // namespace

hipError_t launch_plan(const ckm_graph& g, const Layout& L, const uint64_t* d_S, const uint64_t* d_R,
                       uint32_t flags, int32_t* d_P, int64_t capacity, int64_t* d_count, int64_t* d_mem,
                       int32_t* d_status, char* work, hipStream_t stream) {
  const uint32_t* S = reinterpret_cast<const uint32_t*>(d_S);
  const uint32_t* R = reinterpret_cast<const uint32_t*>(d_R);
  int64_t* cnt = at<int64_t>(work, L.plan_cnt_off);
  int64_t* comp = at<int64_t>(work, L.plan_comp_off);
  int32_t* err = at<int32_t>(work, L.plan_err_off);
  int64_t* off = at<int64_t>(work, L.plan_pos_off);
  int64_t* rbase = at<int64_t>(work, L.plan_rbase_off);
  int32_t* go = at<int32_t>(work, L.plan_go_off);
  hipLaunchKernelGGL(ckm_plan_count_kernel, dim3(g.n), dim3(kPlanWave), 0, stream, g.n, L.row_words, S, R,
                     g.d_dep_ptr, g.d_dep_idx, cnt, comp, err);
  hipLaunchKernelGGL(ckm_plan_scan_kernel, dim3(1), dim3(kScanThreads), 0, stream, g.n,
                     static_cast<const int64_t*>(cnt), static_cast<const int64_t*>(comp),
                     static_cast<const int32_t*>(err), off, rbase, capacity, d_P ? 1 : 0, d_count, d_status, go);
  if (d_P) {
    PlanArgs a;
    a.n = g.n;
    a.rw = L.row_words;
    a.early = (flags & CKM_PLAN_EARLY_FREE) ? 1 : 0;
    a.base = g.base;
    a.S = S;
    a.R = R;
    a.dep_ptr = g.d_dep_ptr;
    a.dep_idx = g.d_dep_idx;
    a.user_ptr = g.d_user_ptr;
    a.user_idx = g.d_user_idx;
    a.M = g.d_M;
    a.off = off;
    a.rbase = rbase;
    a.go = go;
    a.P = d_P;
    a.mem = d_mem;
    a.capacity = capacity;
    hipLaunchKernelGGL(ckm_plan_emit_kernel, dim3(g.n), dim3(kPlanWave), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace ckm
