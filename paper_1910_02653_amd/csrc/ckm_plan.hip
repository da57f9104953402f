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
// Inclusive prefix sums over the lanes of the wave.
__device__ __forceinline__ int64_t wave_scan_i64(int64_t x, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(x, o);
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
                                                                   int32_t* __restrict__ err,
                                                                   int32_t* __restrict__ rpre) {
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
  // computes of R_t before each word, for the registers of later stages
  {
    int64_t carry = 0;
    for (int w0 = 0; w0 < nwt; w0 += kPlanWave) {
      const int w = w0 + lane;
      const int64_t pc = w < nwt ? __popc(r_word(R, rw, t, w)) : 0;
      const int64_t inc = wave_scan_i64(pc, lane);
      if (w < nwt) rpre[(size_t)t * kMaxNodesWords + w] = (int32_t)(carry + inc - pc);
      carry += __shfl(inc, kPlanWave - 1);
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
  int32_t rtw;                       // words per column of RT: ceil(n / 32)
  int64_t base;                      // M_in + 2 M_param
  const uint32_t* S;
  const uint32_t* R;
  const uint32_t* RT;                // R transposed: bit s of RT[i] = R[s][i]
  const int32_t* rpre;               // [n][kMaxNodesWords]: computes in row s before word w
  const int32_t* dep_ptr;
  const int32_t* dep_idx;
  const int32_t* user_ptr;
  const int32_t* user_idx;
  const int64_t* M;
  const int64_t* off;
  const int64_t* rbase;
  const int32_t* go;
  int32_t* P;                        // [capacity][4]: op, node, register, stage
  int64_t* mem;                      // [capacity] or null
  int64_t capacity;
};

__device__ __forceinline__ void put_stmt(const PlanArgs& a, int64_t s, int op, int node, int64_t reg, int t,
                                         int64_t mem_after) {
  // positions come from the count kernel's totals, which the scan checked
  // against the capacity; the guard keeps every store inside the buffers
  if (s < 0 || s >= a.capacity) return;
  int32_t* p = a.P + 4 * s;
  p[0] = op;
  p[1] = node;
  p[2] = (int32_t)reg;
  p[3] = t;
  if (a.mem) a.mem[s] = mem_after;
}

// Register of value i live in stage t: computed in this stage, or else kept
// from the last stage s < t that computed it (R[s][i] = 1; no value is both
// kept and recomputed, so the kept copy is that one). s is the highest set
// bit below t of column i of R.
__device__ int64_t reg_of(const PlanArgs& a, int t, int i, const uint32_t* rt_l, const int32_t* wpre) {
  const int w = i >> 5;
  const uint32_t below = (1u << (i & 31)) - 1u;
  if (bit_of(rt_l[w], i)) return a.rbase[t] + wpre[w] + __popc(rt_l[w] & below);
  const uint32_t* col = a.RT + (size_t)i * a.rtw;
  int sw = (t - 1) >> 5;
  const int top = (t - 1) & 31;
  uint32_t m = col[sw] & (top == 31 ? ~0u : ((2u << top) - 1u));
  while (m == 0u && sw > 0) m = col[--sw];
  if (m == 0u) return -1;   // unreachable for a checked schedule
  const int s = 32 * sw + 31 - __clz(m);
  return a.rbase[s] + a.rpre[(size_t)s * kMaxNodesWords + w] + __popc(r_word(a.R, a.rw, s, w) & below);
}

// Column words of RT: block (node group of 64, stage word); lane = node.
__global__ void __launch_bounds__(kPlanWave) ckm_plan_transpose_kernel(int32_t n, int32_t rw,
                                                                       const uint32_t* __restrict__ R,
                                                                       int32_t rtw, uint32_t* __restrict__ RT) {
  const int i = blockIdx.x * kPlanWave + threadIdx.x;
  const int sw = blockIdx.y;
  uint32_t word = 0;
  for (int q = 0; q < 32; ++q) {
    const int s = 32 * sw + q;
    if (s < n && i < n) word |= bit_of(r_word(R, rw, s, i >> 5), i) << q;
  }
  if (i < n) RT[(size_t)i * rtw + sw] = word;
}

constexpr int kMaxChunks = CKM_MAX_NODES / kPlanWave;

// Stage t = n - 1 - blockIdx.x (longest first): kEmitWaves waves (4, or 16
// for large graphs, whose LDS allows only a few blocks per CU). Node k's
// statements are its compute and the deallocations whose free point is k;
// an unused checkpoint's deallocation sits at the stage start or end.
//   1. free point of every node (LDS), unused checkpoints per 64 nodes, the
//      stage's starting memory U_{t,0};
//   2. per node: statement count and memory change (LDS), per 64 nodes the
//      totals;
//   3. one wave: offsets of every 64-node group (positions and memory);
//   4. every wave writes the statements of its groups.
// Dynamic LDS: n int64 (memory change), then n + n int32 (free point,
// statement count).
template <int kEmitWaves>
__global__ void __launch_bounds__(kEmitWaves * kPlanWave) ckm_plan_emit_kernel(PlanArgs a) {
  constexpr int kEmitThreads = kEmitWaves * kPlanWave;
  extern __shared__ int64_t dyn[];
  __shared__ uint32_t st_l[kMaxNodesWords], rt_l[kMaxNodesWords], sn_l[kMaxNodesWords];
  __shared__ int32_t wpre[kMaxNodesWords];
  __shared__ int64_t ch_cnt[kMaxChunks], uc_cnt[kMaxChunks];
  __shared__ int64_t ch_mem[kMaxChunks], uc_mem[kMaxChunks];
  __shared__ int64_t kept_part[kEmitWaves];
  int64_t* cmem = dyn;
  int32_t* fpt = reinterpret_cast<int32_t*>(dyn + a.n);
  int32_t* ccnt = fpt + a.n;
  const int t = a.n - 1 - (int)blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & (kPlanWave - 1);
  const int wave = tid / kPlanWave;
  if (a.go[0] == 0) return;
  const int nwt = (t >> 5) + 1;
  const int nc = (t >> 6) + 1;
  for (int w = tid; w < nwt; w += kEmitThreads) {
    st_l[w] = s_word(a.S, a.rw, t, w);
    rt_l[w] = r_word(a.R, a.rw, t, w);
    sn_l[w] = (t + 1 < a.n) ? s_word(a.S, a.rw, t + 1, w) : 0u;
  }
  __syncthreads();
  if (wave == 0) {   // computes in R_t before each word (<= 128 words)
    int64_t carry = 0;
    for (int w0 = 0; w0 < nwt; w0 += kPlanWave) {
      const int w = w0 + lane;
      const int64_t c = w < nwt ? __popc(rt_l[w]) : 0;
      const int64_t inc = wave_scan_i64(c, lane);
      if (w < nwt) wpre[w] = (int32_t)(carry + inc - c);
      carry += __shfl(inc, kPlanWave - 1);
    }
  }
  // 1. free points; wave w owns the 64-node groups w, w + 4, ...
  int64_t kept_bytes = 0;
  for (int c = wave; c < nc; c += kEmitWaves) {
    const int i = 64 * c + lane;
    int f = kFreeNone;
    int64_t mi = 0;
    if (i <= t) {
      const uint32_t si = bit_of(st_l[i >> 5], i), ri = bit_of(rt_l[i >> 5], i);
      mi = a.M[i];
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
      if (si) kept_bytes += mi;
    }
    const bool un = f == kFreeUnused;
    const int64_t su = wave_sum_i64(un ? -mi : 0);
    const uint64_t um = __ballot(un);
    if (lane == 0) {
      uc_cnt[c] = __popcll(um);
      uc_mem[c] = su;
    }
  }
  kept_bytes = wave_sum_i64(kept_bytes);
  if (lane == 0) kept_part[wave] = kept_bytes;
  __syncthreads();
  // 2. per node: statements and memory change
  for (int c = wave; c < nc; c += kEmitWaves) {
    const int k = 64 * c + lane;
    int64_t cn = 0;
    int64_t d = 0;
    if (k <= t) {
      if (bit_of(rt_l[k >> 5], k)) {
        cn = 1;
        d = a.M[k];
      }
      for (int e = a.dep_ptr[k]; e < a.dep_ptr[k + 1]; ++e) {
        const int i = a.dep_idx[e];
        if (fpt[i] == k) {
          ++cn;
          d -= a.M[i];
        }
      }
      if (fpt[k] == k) {
        ++cn;
        d -= a.M[k];
      }
      ccnt[k] = (int32_t)cn;
      cmem[k] = d;
    }
    cn = wave_sum_i64(cn);
    d = wave_sum_i64(d);
    if (lane == 0) {
      ch_cnt[c] = cn;
      ch_mem[c] = d;
    }
  }
  __syncthreads();
  // 3. offsets of the groups (nc <= 64: one wave)
  if (wave == 0) {
    int64_t u0 = a.base;
    for (int w = 0; w < kEmitWaves; ++w) u0 += kept_part[w];
    const bool in = lane < nc;
    const int64_t cn = in ? ch_cnt[lane] : 0, un = in ? uc_cnt[lane] : 0;
    const int64_t dm = in ? ch_mem[lane] : 0, um = in ? uc_mem[lane] : 0;
    const int64_t cn_inc = wave_scan_i64(cn, lane), un_inc = wave_scan_i64(un, lane);
    const int64_t dm_inc = wave_scan_i64(dm, lane), um_inc = wave_scan_i64(um, lane);
    const int64_t node_total = __shfl(cn_inc, kPlanWave - 1), un_total = __shfl(un_inc, kPlanWave - 1);
    const int64_t node_mem = __shfl(dm_inc, kPlanWave - 1), un_mem = __shfl(um_inc, kPlanWave - 1);
    const int64_t o = a.off[t];
    int64_t node_pos = o, un_pos = o + node_total;
    int64_t node_mb = u0, un_mb = u0 + node_mem;
    if (a.early) {
      un_pos = o;
      un_mb = u0;
      node_pos = o + un_total;
      node_mb = u0 + un_mem;
    }
    if (in) {
      ch_cnt[lane] = node_pos + cn_inc - cn;
      ch_mem[lane] = node_mb + dm_inc - dm;
      uc_cnt[lane] = un_pos + un_inc - un;
      uc_mem[lane] = un_mb + um_inc - um;
    }
  }
  __syncthreads();
  // 4. statements
  for (int c = wave; c < nc; c += kEmitWaves) {
    const int k = 64 * c + lane;
    const bool in = k <= t;
    const int64_t cn = in ? ccnt[k] : 0;
    const int64_t d = in ? cmem[k] : 0;
    const int64_t cinc = wave_scan_i64(cn, lane);
    const int64_t dinc = wave_scan_i64(d, lane);
    int64_t s = ch_cnt[c] + cinc - cn;
    int64_t mu = ch_mem[c] + dinc - d;   // memory before node k's statements
    if (cn) {
      if (bit_of(rt_l[k >> 5], k)) {
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
    // unused checkpoints of this group, ascending
    const bool un = in && fpt[k] == kFreeUnused;
    const uint64_t um = __ballot(un);
    if (um) {
      const int64_t du = un ? -a.M[k] : 0;
      const int64_t uinc = wave_scan_i64(du, lane);
      if (un)
        put_stmt(a, uc_cnt[c] + __popcll(um & ((1ull << lane) - 1ull)), 1, k, reg_of(a, t, k, rt_l, wpre), t,
                 uc_mem[c] + uinc);
    }
  }
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
  int32_t* rpre = at<int32_t>(work, L.plan_rpre_off);
  uint32_t* RT = at<uint32_t>(work, L.plan_rt_off);
  const int32_t rtw = (g.n + 31) / 32;
  hipLaunchKernelGGL(ckm_plan_count_kernel, dim3(g.n), dim3(kPlanWave), 0, stream, g.n, L.row_words, S, R,
                     g.d_dep_ptr, g.d_dep_idx, cnt, comp, err, rpre);
  hipLaunchKernelGGL(ckm_plan_scan_kernel, dim3(1), dim3(kScanThreads), 0, stream, g.n,
                     static_cast<const int64_t*>(cnt), static_cast<const int64_t*>(comp),
                     static_cast<const int32_t*>(err), off, rbase, capacity, d_P ? 1 : 0, d_count, d_status, go);
  if (d_P) {
    hipLaunchKernelGGL(ckm_plan_transpose_kernel, dim3((g.n + kPlanWave - 1) / kPlanWave, rtw), dim3(kPlanWave),
                       0, stream, g.n, L.row_words, R, rtw, RT);
    PlanArgs a;
    a.n = g.n;
    a.rw = L.row_words;
    a.early = (flags & CKM_PLAN_EARLY_FREE) ? 1 : 0;
    a.rtw = rtw;
    a.base = g.base;
    a.S = S;
    a.R = R;
    a.RT = RT;
    a.rpre = rpre;
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
    const size_t lds = (size_t)g.n * (sizeof(int64_t) + 2 * sizeof(int32_t));
    const bool wide = g.n > 1024;
    void (*fn)(PlanArgs) = wide ? ckm_plan_emit_kernel<16> : ckm_plan_emit_kernel<4>;
    hipError_t e = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(g.n), dim3((wide ? 16 : 4) * kPlanWave), lds, stream, a);
  }
  return hipGetLastError();
}

}  // namespace ckm
