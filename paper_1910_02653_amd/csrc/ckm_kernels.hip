// HIP kernels for gfx950: batched rounding, Algorithm 2 repair, memory
// simulation, reduction and argmin of Checkmate candidate schedules.
//
// Work decomposition: one wave of 64 lanes owns 64 candidates (lane =
// candidate) and one work item of stages. All lanes walk the same nodes in
// the same order, so graph data and loop bounds are wave-uniform and only the
// candidates' bits and running sums differ per lane. Three evaluate kernels
// share that shape:
// - ckm_mask_eval_kernel and ckm_seen_eval_kernel (graphs up to 4096 nodes
//   with the row arrays in the work buffer): S is rounded beforehand into
//   mask rows, one 64-bit word per (row, node) whose bit j is candidate j of
//   the group, so the repair and the FREE tests are 64-bit scalar operations
//   for the whole group and only the binary64 sums run per lane;
// - ckm_eval_kernel (the rest: larger or wide graphs, no row arrays): each
//   lane keeps its own bit rows (32-bit words, bit i%32 of word i/32): S_t,
//   which becomes R_t as the scan passes, in LDS laid out [word][lane] so that
//   a wave-uniform word index touches 64 consecutive dwords, and S_{t+1} in
//   vector registers (in LDS too for the largest graphs). S rows come from a
//   row array in HBM, [row][word][candidate], or are made in the kernel.
//
// Sums of sizes and costs run in binary64 while the graph's totals stay below
// 2^53, so every partial sum is an exactly represented integer and the result
// is identical to int64 arithmetic in any order; a graph whose totals reach
// 2^53 (a wide graph) is summed in int64 by ckm_eval_kernel.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstddef>
#include <cmath>
#include <cstdint>
#include <cstring>

#include "ckm_internal.h"


namespace ckm {
namespace {

// Read-only data that every lane of a wave reads at the same address (graph
// CSR, sizes, thresholds): load it through the constant address space so
// that uniform reads become scalar loads through the scalar cache.
template <typename T>
using cptr = const __attribute__((address_space(4))) T*;

template <typename T>
__host__ __device__ __forceinline__ cptr<T> as_const(const T* p) {
  return (cptr<T>)(p);
}

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): multipliers for counter
// words 0 and 2, key advanced by the Weyl constants between rounds.
constexpr uint32_t kPhiloxM0 = 0xD2511F53u;
constexpr uint32_t kPhiloxM1 = 0xCD9E8D57u;
constexpr uint32_t kPhiloxW0 = 0x9E3779B9u;
constexpr uint32_t kPhiloxW1 = 0xBB67AE85u;

// a ^ b ^ c in one VALU instruction (c is wave-uniform: the round key).
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);  // truth table of a ^ b ^ c
}

__device__ __forceinline__ void philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                              uint32_t k0, uint32_t k1, uint32_t x[4]) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)kPhiloxM0 * c0;
    const uint64_t p1 = (uint64_t)kPhiloxM1 * c2;
    const uint32_t n0 = xor3((uint32_t)(p1 >> 32), c1, k0);
    const uint32_t n2 = xor3((uint32_t)(p0 >> 32), c3, k1);
    c0 = n0;
    c1 = (uint32_t)p1;
    c2 = n2;
    c3 = (uint32_t)p0;
    k0 += kPhiloxW0;
    k1 += kPhiloxW1;
  }
  x[0] = c0; x[1] = c1; x[2] = c2; x[3] = c3;
}

// word = 2^8 word + (8 rounding bits), high draw first: bit j of the new
// byte is [u_j < q_j], where u_j is 16-bit half (j mod 2) of x[j / 2] and
// q_j is wave-uniform. Each compare writes a lane mask that a carry-in add
// folds into the word; three masks rotate so that every add reads a mask
// written at least two instructions earlier (the VALU-written SGPR to VALU
// lane-mask read distance).
__device__ __forceinline__ uint32_t append8_uniform(uint32_t word, const uint32_t x[4], const uint32_t q[8]) {
  uint64_t m0, m1, m2;
  asm("v_cmp_lt_u32_sdwa %[m0], %[x3], %[q7] src0_sel:WORD_1 src1_sel:DWORD\n\t"
      "v_cmp_lt_u32_sdwa %[m1], %[x3], %[q6] src0_sel:WORD_0 src1_sel:DWORD\n\t"
      "v_cmp_lt_u32_sdwa %[m2], %[x2], %[q5] src0_sel:WORD_1 src1_sel:DWORD\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m0]\n\t"
      "v_cmp_lt_u32_sdwa %[m0], %[x2], %[q4] src0_sel:WORD_0 src1_sel:DWORD\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m1]\n\t"
      "v_cmp_lt_u32_sdwa %[m1], %[x1], %[q3] src0_sel:WORD_1 src1_sel:DWORD\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m2]\n\t"
      "v_cmp_lt_u32_sdwa %[m2], %[x1], %[q2] src0_sel:WORD_0 src1_sel:DWORD\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m0]\n\t"
      "v_cmp_lt_u32_sdwa %[m0], %[x0], %[q1] src0_sel:WORD_1 src1_sel:DWORD\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m1]\n\t"
      "v_cmp_lt_u32_sdwa %[m1], %[x0], %[q0] src0_sel:WORD_0 src1_sel:DWORD\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m2]\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m0]\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m1]"
      : [w] "+v"(word), [m0] "=&s"(m0), [m1] "=&s"(m1), [m2] "=&s"(m2)
      : [x0] "v"(x[0]), [x1] "v"(x[1]), [x2] "v"(x[2]), [x3] "v"(x[3]), [q0] "s"(q[0]), [q1] "s"(q[1]),
        [q2] "s"(q[2]), [q3] "s"(q[3]), [q4] "s"(q[4]), [q5] "s"(q[5]), [q6] "s"(q[6]), [q7] "s"(q[7])
      : "vcc");
  return word;
}

// Same bits, thresholds in any register class.
__device__ __forceinline__ uint32_t append8(uint32_t word, const uint32_t x[4], const uint32_t q[8]) {
#pragma unroll
  for (int j = 7; j >= 0; --j) {
    const uint32_t u = (x[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
    word = word + word + (u < q[j] ? 1u : 0u);
  }
  return word;
}

// 32 rounding decisions of row r, candidate k: bits i = 32w .. 32w+31 of
// S_k[r] (Section 5.1 randomized rounding, thresholds q). Entries i >= r
// have q = 0 and round to 0. The word is assembled high bit first.
// kUniformQ: the row pointer and w are the same for the whole wave.
template <bool kUniformQ, typename QPtr>
__device__ __forceinline__ uint32_t round_word(QPtr qrow, int w, int r, uint32_t k, uint32_t key0,
                                               uint32_t key1) {
  uint32_t word = 0;
#pragma unroll
  for (int b = 3; b >= 0; --b) {
    const int m = 4 * w + b;        // draws 8m .. 8m+7 share one Philox output
    if (8 * m >= r) {               // this part of the word is beyond the row
      word <<= 8;
      continue;
    }
    uint32_t x[4], q[8];
    philox4x32_10((uint32_t)m, (uint32_t)r, k, 0u, key0, key1, x);
#pragma unroll
    for (int j = 0; j < 8; ++j) q[j] = qrow[8 * m + j];
    word = kUniformQ ? append8_uniform(word, x, q) : append8(word, x, q);
  }
  return word;
}

// word = 2^8 word + (8 threshold bits), high bit first: bit j of the new byte
// is [rk < q_j] with rk the lane's threshold rank and q_j wave-uniform keys
// (same carry-in fold as append8_uniform).
__device__ __forceinline__ uint32_t append8_rank(uint32_t word, uint32_t rk, const uint32_t q[8]) {
  uint64_t m0, m1, m2;
  asm("v_cmp_lt_u32_e64 %[m0], %[rk], %[q7]\n\t"
      "v_cmp_lt_u32_e64 %[m1], %[rk], %[q6]\n\t"
      "v_cmp_lt_u32_e64 %[m2], %[rk], %[q5]\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m0]\n\t"
      "v_cmp_lt_u32_e64 %[m0], %[rk], %[q4]\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m1]\n\t"
      "v_cmp_lt_u32_e64 %[m1], %[rk], %[q3]\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m2]\n\t"
      "v_cmp_lt_u32_e64 %[m2], %[rk], %[q2]\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m0]\n\t"
      "v_cmp_lt_u32_e64 %[m0], %[rk], %[q1]\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m1]\n\t"
      "v_cmp_lt_u32_e64 %[m1], %[rk], %[q0]\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m2]\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m0]\n\t"
      "v_addc_co_u32 %[w], vcc, %[w], %[w], %[m1]"
      : [w] "+v"(word), [m0] "=&s"(m0), [m1] "=&s"(m1), [m2] "=&s"(m2)
      : [rk] "v"(rk), [q0] "s"(q[0]), [q1] "s"(q[1]), [q2] "s"(q[2]), [q3] "s"(q[3]), [q4] "s"(q[4]),
        [q5] "s"(q[5]), [q6] "s"(q[6]), [q7] "s"(q[7])
      : "vcc");
  return word;
}

// 32 threshold-rounding decisions of row r: bits i = 32w .. 32w+31 of
// S[r][i] = [clamp(S*[r][i], 0, 1) > p_k], computed exactly as [rk < key[r][i]]
// with key = #{j : p_j < clamp(S*)} and rk = #{j : p_j < p_k}. Keys of
// entries i >= r are 0. kUniformQ: the row pointer and w are wave-uniform.
template <bool kUniformQ, typename QPtr>
__device__ __forceinline__ uint32_t threshold_word(QPtr qrow, int w, int r, uint32_t rk) {
  uint32_t word = 0;
#pragma unroll
  for (int b = 3; b >= 0; --b) {
    const int m = 4 * w + b;
    if (8 * m >= r) {
      word <<= 8;
      continue;
    }
    uint32_t q[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) q[j] = qrow[8 * m + j];
    if (kUniformQ) {
      word = append8_rank(word, rk, q);
    } else {
#pragma unroll
      for (int j = 7; j >= 0; --j) word = word + word + (rk < q[j] ? 1u : 0u);
    }
  }
  return word;
}

// ---------------------------------------------------------------------------
// Per-node record, read once per node visit. Masks are relative to the node
// v: bit d <-> node v + 1 + d, d < 32 (the scan's window of R bits). A
// reference locates one bit of a row: its word index (8 bits, packed four to
// a dword) and its bit position (5 bits, packed six to a dword). The
// references are: the user of v beyond v + 32 in the R row (fu), and per
// dependency slot the user of the dep beyond v + 32 in the R row (fl) and
// the dep in the next-stage checkpoint row (s1); absent ones point at node
// n, whose bit no row ever sets.
constexpr int kRecDeps = 4;
struct NodeRec {
  uint64_t M, C;            // M_v, C_v (binary64, or int64 for a wide graph)
  uint32_t umask;           // users u of v with u <= v + 32
  uint32_t refs0;           // word indices: fu | fl0 << 8 | s1_0 << 16 | fl1 << 24
  uint32_t refs1;           // s1_1 word | deps << 8 | slow << 11 | bit positions 6-8 at 12, 17, 22
  uint32_t bits0;           // bit positions 0-5 (fu, s1_0, fl0, s1_1, fl1, s1_2) | min(deps, 3) << 30,
                            // or 3 << 30 for a node outside the format
  uint32_t lm[kRecDeps];    // per slot: users u of the dep with v < u <= v + 32
  uint32_t refs2;           // word indices: fl2 | s1_2 << 8 | fl3 << 16 | s1_3 << 24
  uint32_t pad0;
  uint64_t dM[kRecDeps];    // M of each dependency slot
  uint32_t pad1[2];
  // fp64 operands again, read by two wave-uniform 16-byte loads: M_v, C_v,
  // and the M of dependency slots 0 and 1
  uint64_t mc[2], dm01[2];
  uint32_t pad[32];         // one dword per lane of a 64-lane load
};
static_assert(sizeof(NodeRec) == kNodeRecBytes, "node record layout");
static_assert(offsetof(NodeRec, mc) % 16 == 0 && offsetof(NodeRec, dm01) % 16 == 0, "16-byte loads");
// Dword indices of the fields that move to scalar registers (v_readlane).
constexpr int kDwUmask = 4, kDwRefs0 = 5, kDwRefs1 = 6, kDwBits0 = 7, kDwLm = 8, kDwRefs2 = 12, kDwDM = 14;
static_assert(offsetof(NodeRec, umask) == 4 * kDwUmask && offsetof(NodeRec, refs0) == 4 * kDwRefs0 &&
                  offsetof(NodeRec, refs1) == 4 * kDwRefs1 && offsetof(NodeRec, bits0) == 4 * kDwBits0 &&
                  offsetof(NodeRec, lm) == 4 * kDwLm && offsetof(NodeRec, refs2) == 4 * kDwRefs2 &&
                  offsetof(NodeRec, dM) == 4 * kDwDM,
              "dword indices used by RecRegs, issue_reads and the closure kernel");
constexpr uint32_t kRefsSlow = 1u << 11;   // refs1: node does not fit the record format

// A slow node (more than four dependencies, or more than one user beyond
// v + 32, for v or for one of its dependencies) reads only umask, refs0,
// refs1, bits0 and the fp64 groups of its record. The other dwords then hold
// its lists in a second form:
//   dword 32: far users of v (count) | dependencies (count) << 8 | kExtValid
//   dwords 33-39: v's users beyond v + 32 (node numbers, two 16-bit fields
//     per dword)
//   dependency slot d at dwords ext_slot(d) ..+5: the dependency's users u
//     with v < u <= v + 32 as a mask (bit u - v - 1); M of the dependency
//     (binary64, two dwords); its node number | the count of its users beyond
//     v + 32 << 16; those users (two dwords, two per dword)
// A node beyond these counts walks the CSR lists (dword 32 without kExtValid).
constexpr int kDwExt = 32, kExtFar = 14, kExtDeps = 6, kExtLate = 4;
constexpr uint32_t kExtValid = 1u << 31;
__host__ __device__ constexpr int ext_slot(int d) { return d < 4 ? 40 + 6 * d : 8 + 6 * (d - 4); }
static_assert(ext_slot(3) + 6 <= 64 && ext_slot(5) + 6 <= 24 && kDwExt + 1 + kExtFar / 2 <= ext_slot(0),
              "extended form inside the record, clear of the fields a slow node reads");
static_assert(offsetof(NodeRec, mc) >= 24 * 4 && offsetof(NodeRec, dm01) + 16 <= 32 * 4, "fp64 groups at 24-31");

__device__ __forceinline__ double dbl(uint32_t lo, uint32_t hi) {
  return __hiloint2double((int)hi, (int)lo);
}

// max(a, b) for values that are never NaN, without the quieting step that
// fmax adds on a loop-carried operand.
__device__ __forceinline__ double max_f64(double a, double b) {
  double d;
  asm("v_max_f64 %0, %1, %2" : "=v"(d) : "v"(a), "v"(b));
  return d;
}

// The sums of the scan: binary64, exact while every partial sum stays below
// 2^53 (the host checks the graph's totals), or int64 for a wide graph. The
// b01 arguments are 0 or 1. In int64 the stage peak U0 - Y + max is formed
// with wrapping additions: its terms may leave the int64 range on the way,
// the result (a memory level of the stage) does not.
template <bool kWide> struct Ar;
template <> struct Ar<false> {
  using T = double;
  static __device__ T of(uint32_t lo, uint32_t hi) { return dbl(lo, hi); }
  static __device__ T of_i(int64_t x) { return (double)x; }
  static __device__ T madd(T acc, uint32_t b01, T m) { return fma((double)b01, m, acc); }
  static __device__ T msub(T acc, uint32_t b01, T m) { return fma(-(double)b01, m, acc); }
  static __device__ T max(T a, T b) { return max_f64(a, b); }
  static __device__ T lowest() { return -INFINITY; }
  static __device__ T stage_peak(T U0, T Y, T m) { return U0 - Y + m; }
  static __device__ T seg_max(T a, T b) { return fmax(a, b); }
  static __device__ int64_t i64(T x) { return (int64_t)x; }
};
template <> struct Ar<true> {
  using T = int64_t;
  static __device__ T of(uint32_t lo, uint32_t hi) { return (int64_t)(((uint64_t)hi << 32) | lo); }
  static __device__ T of_i(int64_t x) { return x; }
  static __device__ T madd(T acc, uint32_t b01, T m) { return acc + (m & -(int64_t)b01); }
  static __device__ T msub(T acc, uint32_t b01, T m) { return acc - (m & -(int64_t)b01); }
  static __device__ T max(T a, T b) { return a > b ? a : b; }
  static __device__ T lowest() { return INT64_MIN; }
  static __device__ T stage_peak(T U0, T Y, T m) { return (int64_t)((uint64_t)U0 - (uint64_t)Y + (uint64_t)m); }
  static __device__ T seg_max(T a, T b) { return a > b ? a : b; }
  static __device__ int64_t i64(T x) { return x; }
};


// A node record spread over the lanes of one vector register: lane L holds
// dword L. Fields are moved to scalar registers when used
// (v_readlane), so a record costs 256 bytes of vector-memory return per
// wave instead of 128 bytes for each of the 64 lanes.
struct RecRegs {
  uint32_t w;
  uint4 mc, dm;  // M_v, C_v and the M of slots 0-1, in every lane
  __device__ uint32_t get(int i) const { return __builtin_amdgcn_readlane(w, i); }
  template <bool W> __device__ typename Ar<W>::T M() const { return Ar<W>::of(mc.x, mc.y); }
  template <bool W> __device__ typename Ar<W>::T C() const { return Ar<W>::of(mc.z, mc.w); }
  template <bool W> __device__ typename Ar<W>::T dM01(int s) const {
    return s == 0 ? Ar<W>::of(dm.x, dm.y) : Ar<W>::of(dm.z, dm.w);
  }
  __device__ uint32_t umask() const { return get(kDwUmask); }
  __device__ uint32_t refs0() const { return get(kDwRefs0); }
  __device__ uint32_t refs1() const { return get(kDwRefs1); }
  __device__ uint32_t bits0() const { return get(kDwBits0); }
  __device__ uint32_t lm(int s) const { return get(kDwLm + s); }
  __device__ uint32_t refs2() const { return get(kDwRefs2); }
  template <bool W> __device__ typename Ar<W>::T dM(int s) const {
    return Ar<W>::of(get(kDwDM + 2 * s), get(kDwDM + 1 + 2 * s));
  }
};

// Bit position k of a record (0: fu; 1 + 2s: s1 of slot s; 2 + 2s: fl of
// slot s) from bits0 and refs1; only the low five bits of the result matter
// to the bit-field extracts that use it.
__device__ __forceinline__ uint32_t bitpos(uint32_t b0, uint32_t refs1, int k) {
  return k < 6 ? (b0 >> (5 * k)) : (refs1 >> (12 + 5 * (k - 6)));
}

// Word index of byte j of a packed dword of word indices.
__device__ __forceinline__ uint32_t word_at(uint32_t refs, int j) { return (refs >> (8 * j)) & 0xFFu; }

// Buffer descriptor word 3 for raw byte-addressed buffers on gfx9-family
// GPUs (32-bit data format); the hardware returns 0 for reads past the
// record count instead of faulting.
constexpr int kBufWord3 = 0x00020000;

// A node record is loaded in two parts: the lane's dword of it (the fields
// that go to scalar registers; needed one node before the node itself, for
// its LDS reads) and the two fp64 groups, the same 16 bytes in every lane
// (needed when the node is evaluated). These are vector-memory loads, whose
// completion counter is in order, so they can run nodes ahead of their use
// (a scalar load would share its counter with LDS reads). As buffer loads
// with the node's offset in a scalar register they need no per-node address
// arithmetic in vector registers, which a global load of a uniform address
// would (a zero or 64-bit address register rebuilt for each node).
struct RecF {
  uint4 mc, dm;
};
__device__ __forceinline__ void load_rec_w(uint32_t& w, __amdgpu_buffer_rsrc_t rs, int v) {
  const int so = __builtin_amdgcn_readfirstlane(v) * kNodeRecBytes;
  w = __builtin_amdgcn_raw_buffer_load_b32(rs, (threadIdx.x & 63u) * 4u, so, 0);
}
__device__ __forceinline__ void load_rec_f(RecF& f, __amdgpu_buffer_rsrc_t rs, int v) {
  const int so = __builtin_amdgcn_readfirstlane(v) * kNodeRecBytes;
  const auto mc = __builtin_amdgcn_raw_buffer_load_b128(rs, 0, so + (int)offsetof(NodeRec, mc), 0);
  const auto dm = __builtin_amdgcn_raw_buffer_load_b128(rs, 0, so + (int)offsetof(NodeRec, dm01), 0);
  f.mc = make_uint4(mc[0], mc[1], mc[2], mc[3]);
  f.dm = make_uint4(dm[0], dm[1], dm[2], dm[3]);
}

struct EvalArgs {
  int32_t n, K, ldq, det_words, row_words;
  int32_t items, kind, P, T0, R1, R2;   // work plan (see Plan)
  uint32_t key0, key1;
  uint32_t det0;                 // CKM_F_DET0 given
  int64_t base;                  // M_in + 2 M_param
  cptr<uint32_t> q;
  cptr<uint32_t> det;
  cptr<int64_t> M;
  cptr<int32_t> user_ptr;
  cptr<int32_t> user_idx;
  cptr<int32_t> dep_ptr;
  cptr<int32_t> dep_idx;
  cptr<int32_t> dep_upos;
  const uint4* __restrict__ recs;
  const uint32_t* __restrict__ s_user;  // kSrcUser: caller-supplied S rows ([K][n][s_words])
  int32_t s_words;                      // 32-bit words per supplied row
  const uint32_t* __restrict__ rank;    // kSrcThreshold: [K] threshold ranks (q holds the keys)
  const uint32_t* __restrict__ rows;    // kSrcRows: S rows, word w of row t at (row_base(t) + w) * kpad + k
  uint32_t* __restrict__ rrows;         // R rows out, same layout, or NULL
  int32_t kpad;                         // row arrays: candidates per row word (64 * groups)
  int64_t* __restrict__ part_peak;   // [K] running max over work items
  int64_t* __restrict__ part_cost;   // [K] running sum over work items
  int32_t* __restrict__ hdr;
};

// First stage of range s of `parts` ranges over stages 0 .. m-1 with about
// equal sums of stage lengths (stage t touches t + 1 nodes):
// floor(sqrt(m^2 s / parts)).
__device__ __forceinline__ int split_begin(int m, int parts, int s) {
  if (s <= 0) return 0;
  if (s >= parts) return m;
  const uint64_t x = (uint64_t)m * (uint64_t)m * (uint64_t)s / (uint64_t)parts;
  uint64_t r = (uint64_t)sqrt((double)x);
  while (r * r > x) --r;
  while ((r + 1) * (r + 1) <= x) ++r;
  return (int)r;
}

// Stages [t0, t1) of work item `item` (numbered most expensive first).
template <typename Args>
__device__ __forceinline__ void item_range(const Args& a, int item, int& t0, int& t1) {
  if (a.kind == 0) {
    const int s = a.items - 1 - item;
    t0 = split_begin(a.n, a.items, s);
    t1 = split_begin(a.n, a.items, s + 1);
  } else if (item < a.R1) {
    t1 = a.n - a.P * item;
    t0 = max(a.T0, t1 - a.P);
  } else {
    const int s = a.R2 - 1 - (item - a.R1);
    t0 = split_begin(a.T0, a.R2, s);
    t1 = split_begin(a.T0, a.R2, s + 1);
  }
}

// A lane's view of one LDS row buffer: word w at byte (w * 256) of `base`.
struct Row {
  char* base;  // buffer start + 4 * lane
  __device__ uint32_t& word(int w) const { return *reinterpret_cast<uint32_t*>(base + w * 256); }
  __device__ uint32_t at_word(uint32_t w) const {  // wave-uniform word index
    return *reinterpret_cast<const uint32_t*>(base + (w << 8));
  }
};

// A row held in the lane's vector registers instead of LDS (n < 1024): word
// w is register w of the array; a wave-uniform index selects it with
// s_set_gpr_idx. Same interface as Row.
constexpr int kRegRowWords = 32;
typedef uint32_t u32x32 __attribute__((ext_vector_type(kRegRowWords)));
struct RowReg {
  u32x32 w;
  struct WordRef {  // assignable element of the vector
    u32x32& v;
    int i;
    __device__ WordRef& operator=(uint32_t x) {
      v[i] = x;
      return *this;
    }
    __device__ operator uint32_t() const { return v[i]; }
  };
  __device__ WordRef word(int i) { return WordRef{w, i}; }
  __device__ uint32_t at_word(uint32_t i) const { return w[i]; }  // wave-uniform word index
};

// A row of up to 32 * kVecs words (kVecs = 2 or 4) in the lane's vector
// registers: kVecs 32-word vectors, locals of the kernel held here by
// reference. Word w is element w % 32 of vector w / 32: a wave-uniform branch
// picks the vector, s_set_gpr_idx the element. The asm statements keep the
// branches distinct; merged, they would become one access through a phi of
// pointers, and the vectors would move to scratch memory.
template <int kVecs>
struct RowRegV {
  u32x32 &v0, &v1, &v2, &v3;
  __device__ uint32_t at_word(uint32_t i) const {
    const uint32_t q = i >> 5, r = i & 31u;
    uint32_t x;
    if (q == 0) {
      x = v0[r];
      asm("; row word 0" : "+v"(x));
    } else if (kVecs == 2 || q == 1) {
      x = v1[r];
      asm("; row word 1" : "+v"(x));
    } else if (q == 2) {
      x = v2[r];
      asm("; row word 2" : "+v"(x));
    } else {
      x = v3[r];
      asm("; row word 3" : "+v"(x));
    }
    return x;
  }
  __device__ void set(uint32_t i, uint32_t x) const {
    const uint32_t q = i >> 5, r = i & 31u;
    if (q == 0) {
      v0[r] = x;
      asm volatile("; row set 0");
    } else if (kVecs == 2 || q == 1) {
      v1[r] = x;
      asm volatile("; row set 1");
    } else if (q == 2) {
      v2[r] = x;
      asm volatile("; row set 2");
    } else {
      v3[r] = x;
      asm volatile("; row set 3");
    }
  }
  struct WordRef {
    const RowRegV& row;
    uint32_t i;
    __device__ WordRef& operator=(uint32_t x) {
      row.set(i, x);
      return *this;
    }
    __device__ operator uint32_t() const { return row.at_word(i); }
  };
  __device__ WordRef word(int i) const { return WordRef{*this, (uint32_t)i}; }
};

__device__ __forceinline__ uint32_t bit(uint32_t word, int pos) { return (word >> pos) & 1u; }

// (a & b) | c as one VALU instruction (b wave-uniform).
__device__ __forceinline__ uint32_t and_or(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t d;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(d) : "v"(a), "s"(b), "v"(c));
  return d;
}

// min(x, 1): 1 iff x != 0, as one VALU instruction.
__device__ __forceinline__ uint32_t umin1(uint32_t x) {
  uint32_t y;
  asm("v_min_u32 %0, %1, 1" : "=v"(y) : "v"(x));
  return y;
}

// Words before row r in the rounded-row array: sum over r' < r of r'/32 + 1
// (row r' has words 0 .. r'/32).
__host__ __device__ __forceinline__ size_t row_base(int r) {
  const size_t full = (size_t)(r >> 5), rem = (size_t)(r & 31);
  return 32 * full * (full + 1) / 2 + rem * (full + 1);
}

// Rounds every row once for the evaluate kernel's kSrcRows source: block
// (candidate group, row r), lane = candidate. The same bits gen_row would
// produce: randomized rounding (Section 5.1), or the deterministic row for
// candidate 0 under CKM_F_DET0.
__global__ void __launch_bounds__(kWave) ckm_round_rows_kernel(const uint32_t* __restrict__ q,
                                                               const uint32_t* __restrict__ det, int32_t ldq,
                                                               int32_t det_words, uint32_t key0, uint32_t key1,
                                                               uint32_t det0, int32_t kpad,
                                                               uint32_t* __restrict__ rows) {
  const int r = gridDim.y - 1 - blockIdx.y;  // long rows (high r) dispatched first: a shorter tail
  const uint32_t k = blockIdx.x * kWave + threadIdx.x;
  const bool det_lane = det0 && k == 0;
  cptr<uint32_t> qrow = as_const(q) + (size_t)r * ldq;
  const uint32_t* drow = det + (size_t)r * det_words;
  uint32_t* dst = rows + row_base(r) * (size_t)kpad + k;
  const int nw = (r >> 5) + 1;
  for (int w = 0; w < nw; ++w) {
    uint32_t word = round_word<true>(qrow, w, r, k, key0, key1);
    if (det_lane) word = drow[w];
    dst[(size_t)w * kpad] = word;
  }
}

// Threshold rows for the kSrcRows source: block (candidate group, row r),
// lane = candidate with threshold rank rank[k]; the same words gen_row makes
// for kSrcThreshold. Lanes past K take candidate K-1's rank (results unused).
__global__ void __launch_bounds__(kWave) ckm_threshold_rows_kernel(const uint32_t* __restrict__ q, int32_t ldq,
                                                                   const uint32_t* __restrict__ rank, int32_t K,
                                                                   int32_t kpad, uint32_t* __restrict__ rows) {
  const int r = gridDim.y - 1 - blockIdx.y;  // long rows (high r) dispatched first: a shorter tail
  const uint32_t k = blockIdx.x * kWave + threadIdx.x;
  const uint32_t rk = rank[k < (uint32_t)K ? k : (uint32_t)K - 1u];
  cptr<uint32_t> qrow = as_const(q) + (size_t)r * ldq;
  uint32_t* dst = rows + row_base(r) * (size_t)kpad + k;
  const int nw = (r >> 5) + 1;
  for (int w = 0; w < nw; ++w) {
    // the word's 32 keys at once: one wait instead of one per byte (keys on
    // and above the diagonal are 0 and give 0 bits, so no entry is skipped;
    // the key rows are ldq >= 32 * nw entries long)
    uint32_t key[32];
#pragma unroll
    for (int j = 0; j < 32; ++j) key[j] = qrow[32 * w + j];
    uint32_t word = 0;
#pragma unroll
    for (int b = 3; b >= 0; --b) word = append8_rank(word, rk, key + 8 * b);
    dst[(size_t)w * kpad] = word;
  }
}

// The caller's S matrices ([K][n][s_words] 32-bit words) into the kSrcRows
// layout, bits on and above the diagonal cleared: block (candidate group,
// row r) of 256 threads. Reads run along each candidate's row, writes along
// the candidates; an LDS tile [word][candidate] (stride kWave + 1, no bank
// conflicts either way) turns one into the other. Lanes past K copy
// candidate K-1 (results unused).
__global__ void __launch_bounds__(256) ckm_user_rows_kernel(const uint32_t* __restrict__ s_user, int32_t n,
                                                            int32_t K, int32_t s_words, int32_t kpad,
                                                            uint32_t* __restrict__ rows) {
  extern __shared__ uint32_t tile[];
  const int r = gridDim.y - 1 - blockIdx.y;  // long rows (high r) dispatched first: a shorter tail
  const int nw = (r >> 5) + 1;
  const int k0 = blockIdx.x * kWave;
  const int cells = nw * kWave;
  const uint32_t diag = (1u << (r & 31)) - 1u;  // the diagonal's word keeps bits < r
  for (int j = threadIdx.x; j < cells; j += blockDim.x) {
    const int c = j / nw, w = j - c * nw;
    const int k = min(k0 + c, K - 1);
    uint32_t word = s_user[((size_t)k * n + r) * s_words + w];
    if (w == nw - 1) word &= diag;
    tile[w * (kWave + 1) + c] = word;
  }
  __syncthreads();
  uint32_t* dst = rows + row_base(r) * (size_t)kpad + k0;
  for (int j = threadIdx.x; j < cells; j += blockDim.x) {
    const int w = j / kWave, c = j % kWave;
    dst[(size_t)w * kpad + c] = tile[w * (kWave + 1) + c];
  }
}

// Row r of the candidate into words 0 .. r/32, from the source kSrc:
// randomized rounding of S*, the caller's rows (a.s_user), or threshold
// rounding (lane threshold rank rk against the keys in q).
template <int kSrc, typename RowT>
__device__ __forceinline__ void gen_row(const EvalArgs& a, int r, uint32_t k, bool det_lane, uint32_t rk,
                                        RowT& dst) {
  const int nw = (r >> 5) + 1;
  if (r >= a.n) {  // S after the last stage: nothing is kept
    for (int w = 0; w < nw; ++w) dst.word(w) = 0u;
    return;
  }
  if (kSrc == kSrcRows) {
    // rows rounded beforehand: word w of row r for candidate k is at
    // (row_base(r) + w) * kpad + k, contiguous across the wave
    const uint32_t* src = a.rows + row_base(r) * (size_t)a.kpad + k;
    for (int w = 0; w < nw; ++w) dst.word(w) = src[(size_t)w * a.kpad];
    return;
  }
  if (kSrc == kSrcUser) {
    // caller-supplied S: row r of candidate k; bits on or above the diagonal
    // (i >= r) are cleared. Lanes past K read candidate K-1 (results unused).
    const uint32_t kk = k < (uint32_t)a.K ? k : (uint32_t)a.K - 1u;
    const uint32_t* src = a.s_user + ((size_t)kk * a.n + r) * a.s_words;
    for (int w = 0; w < nw; ++w) {
      uint32_t word = src[w];
      if (w == nw - 1) word &= (1u << (r & 31)) - 1u;   // the diagonal's word: keep bits < r
      dst.word(w) = word;
    }
    return;
  }
  cptr<uint32_t> qrow = a.q + (size_t)r * a.ldq;
  if (kSrc == kSrcThreshold) {
    for (int w = 0; w < nw; ++w) dst.word(w) = threshold_word<true>(qrow, w, r, rk);
    return;
  }
  cptr<uint32_t> drow = a.det + (size_t)r * a.det_words;
  // the round keys are rebuilt per row instead of held for the whole kernel
  uint32_t key0 = a.key0, key1 = a.key1;
  asm volatile("" : "+s"(key0), "+s"(key1));
  for (int w = 0; w < nw; ++w) {
    uint32_t word = round_word<true>(qrow, w, r, k, key0, key1);
    if (det_lane) word = drow[w];
    dst.word(w) = word;
  }
}

// R bit of node u for a lane at node v of the right-to-left scan (v < u <= t):
// nodes v+1 .. v+32 are in the window Rwin (bit d <-> node v + 1 + d); a
// farther node lies in a chunk already finished, whose R word is in A.
__device__ __forceinline__ uint32_t r_bit(int u, int v, uint32_t Rwin, Row A) {
  const int d = u - v - 1;
  if (d < 32) return bit(Rwin, d);
  return bit(A.word(u >> 5), u & 31);
}

// Running state of the right-to-left scan of one stage (per lane).
template <typename T>
struct Scan {
  T U0, Y, maxv, cost;
  uint32_t Rwin;       // R bits of the 32 nodes above the current node
  uint32_t w0, w1;     // S_t and S_{t+1} words of the current chunk
};

// LDS words one node reads: the R word of v's user beyond the window, and
// per dependency slot the R word of its user beyond the window and its
// S_{t+1} word, for the first kSlots slots (the others, if any, are read when
// the node is evaluated). Unused slots reference the "none" bit (node n).
template <int kSlots>
struct LdsVals {
  uint32_t fu;
  uint32_t fl[kSlots];
  uint32_t s1[kSlots];
};

// Keeps a group of scalar values together: all of them are computed before
// any use that follows (the v_readlane results then need no wait states).
__device__ __forceinline__ void pin_s(uint32_t a, uint32_t b, uint32_t c) { asm volatile("" ::"s"(a), "s"(b), "s"(c)); }

// Issues the LDS and register-row reads of the node whose record dword
// (this lane's) is w. They are issued one node ahead of their use: the words
// they read are final by then (a user more than 32 nodes above the node lies
// in a chunk above the current one, already finished; S_{t+1} is not written
// during the stage).
template <int kSlots, typename RowB>
__device__ __forceinline__ void issue_reads(uint32_t w, Row A, RowB& B, LdsVals<kSlots>& L) {
  const uint32_t r0 = __builtin_amdgcn_readlane(w, kDwRefs0), r1 = __builtin_amdgcn_readlane(w, kDwRefs1);
  const uint32_t fu = word_at(r0, 0), fl0 = word_at(r0, 1), s10 = word_at(r0, 2);
  const uint32_t fl1 = word_at(r0, 3), s11 = word_at(r1, 0);
  pin_s(fu, fl0, s10);
  pin_s(fl1, s11, r1);
  L.fu = A.at_word(fu);
  L.fl[0] = A.at_word(fl0);
  L.s1[0] = B.at_word(s10);
  L.fl[1] = A.at_word(fl1);
  L.s1[1] = B.at_word(s11);
  // slots 2 and 3 only for the few nodes that use them
  if (kSlots == 4 && __builtin_expect(((r1 >> 8) & 7u) > 2u, 0)) {
    const uint32_t r2 = __builtin_amdgcn_readlane(w, kDwRefs2);
    const uint32_t fl2 = word_at(r2, 0), s12 = word_at(r2, 1), fl3 = word_at(r2, 2), s13 = word_at(r2, 3);
    pin_s(fl2, s12, fl3);
    pin_s(s13, s13, s13);
    L.fl[kSlots - 2] = A.at_word(fl2);
    L.s1[kSlots - 2] = B.at_word(s12);
    L.fl[kSlots - 1] = A.at_word(fl3);
    L.s1[kSlots - 1] = B.at_word(s13);
  }
}

// One node v of stage t. Algorithm 2's repair runs right to left (reverse
// topological order), so every user of v is decided before v: v is computed
// iff it is node t (constraint 4a), or it is not checkpointed and is kept
// for the next stage (1c) or needed by a computed user (1b). The U
// recurrence of Section 4.4 runs in suffix form in the same pass:
//   val_k = sum_{j>=k} freed_j - sum_{j>k} alloc_j,   U_{t,k} = U_end + val_k,
// so the stage peak is U_end + max_k val_k with U_end = U_{t,0} - Y, Y being
// the suffix value after node 0. freed_v collects FREE(t,i,v) M_i over
// i in Deps[v] u {v}: v computed, i not kept, and no computed user of i
// after v. A holds S_t below the current chunk and R_t above it; B holds
// S_{t+1}. Rows are zero beyond their last word, so a reference to a node
// above t (or to node n, "none") reads 0. kFirst: v == t, which is always
// computed and has no computed user in the stage.
template <bool kWide, bool kFirst, int kSlots, typename RowB>
__device__ __forceinline__ void scan_node(const EvalArgs& a, int t, int v, const RecRegs& rec, const LdsVals<kSlots>& L,
                                          Scan<typename Ar<kWide>::T>& sc, Row A, RowB& B) {
  using AR = Ar<kWide>;
  using T = typename AR::T;
  const int jj = v & 31;
  const uint32_t s0 = bit(sc.w0, jj);
  const uint32_t s1 = bit(sc.w1, jj);
  // the node's scalar fields, read together
  const uint32_t um = rec.umask(), b0 = rec.bits0();
  pin_s(um, b0, b0);
  const T Mv = rec.template M<kWide>();
  const T Cv = rec.template C<kWide>();
  uint32_t anyU, r;
  // val = Y + freed_v, accumulated in place (exact integers: any order)
  T val = sc.Y;
  // deps 0-2 from bits0; 3 means "read refs1" (3 or 4 deps, or a slow node)
  uint32_t nd = b0 >> 30, r1 = 0;
  if (__builtin_expect(nd == 3u, 0)) {
    r1 = rec.refs1();
    nd = (r1 & kRefsSlow) ? 15u : ((r1 >> 8) & 7u);
  }
  if (__builtin_expect(nd != 15u, 1)) {
    if (kFirst) {
      anyU = 0;
      r = 1;
    } else {
      const uint32_t far = __builtin_amdgcn_ubfe(L.fu, b0, 1);
      anyU = and_or(sc.Rwin, um, far);
      anyU = umin1(anyU);
      // s0, s1 and anyU are each 0 or 1, so this is one 3-input bit op
      r = (s1 | anyU) & ~s0;
    }
    // FREE(t,v,v): v computed, not kept, no computed user after it. A node
    // other than t is computed only because it is kept (s1) or used (anyU),
    // so only node t can be freed right after it is computed.
    if (kFirst) val = AR::madd(val, ~s1 & 1u, Mv);
    auto slot = [&](int sl, uint32_t flw, uint32_t s1w) {
      const uint32_t lm = rec.lm(sl);
      T dMs;
      if (sl < 2) {
        dMs = rec.template dM01<kWide>(sl);
      } else {
        const uint32_t d_lo = rec.get(kDwDM + 2 * sl), d_hi = rec.get(kDwDM + 1 + 2 * sl);
        pin_s(d_lo, d_hi, d_hi);
        dMs = AR::of(d_lo, d_hi);
      }
      const uint32_t far = __builtin_amdgcn_ubfe(flw, bitpos(b0, r1, 2 + 2 * sl), 1);
      uint32_t later = and_or(sc.Rwin, lm, far);
      later = umin1(later);
      // r and later are 0 or 1: no mask needed
      const uint32_t fr = r & ~__builtin_amdgcn_ubfe(s1w, bitpos(b0, r1, 1 + 2 * sl), 1) & ~later;
      val = AR::madd(val, fr, dMs);
    };
    // most nodes have one or two dependencies
    if (__builtin_expect(nd >= 1, 1)) slot(0, L.fl[0], L.s1[0]);
    if (__builtin_expect(nd >= 2, 1)) slot(1, L.fl[1], L.s1[1]);
    if (__builtin_expect(nd >= 3, 0)) {
      if (kSlots == 4) {
        slot(2, L.fl[kSlots - 2], L.s1[kSlots - 2]);
        if (nd >= 4) slot(3, L.fl[kSlots - 1], L.s1[kSlots - 1]);
      } else {
        // slots 2 and 3 (few nodes here): their words are read now, not pipelined
        const uint32_t r2 = rec.refs2();
        const uint32_t fl2 = A.at_word(word_at(r2, 0)), s12 = B.at_word(word_at(r2, 1));
        slot(2, fl2, s12);
        if (nd >= 4) {
          const uint32_t fl3 = A.at_word(word_at(r2, 2)), s13 = B.at_word(word_at(r2, 3));
          slot(3, fl3, s13);
        }
      }
    }
  } else if (const uint32_t h = rec.get(kDwExt); h & kExtValid) {
    // outside the record format, inside its second form: the same tests with
    // the far references listed there (each read from the R row; a node
    // above t reads 0, as in the record format)
    const uint32_t nfar = h & 0xFFu, nds = (h >> 8) & 0xFFu;
    auto node16 = [&](int dw, uint32_t f) { return (rec.get(dw + (int)(f >> 1)) >> (16 * (f & 1u))) & 0xFFFFu; };
    if (kFirst) {
      anyU = 0;
      r = 1;
      val = AR::madd(val, ~s1 & 1u, Mv);
    } else {
      uint32_t acc = sc.Rwin & um;
      for (uint32_t f = 0; f < nfar; ++f) {
        const uint32_t u = node16(kDwExt + 1, f);
        acc |= bit(A.at_word(u >> 5), u & 31);
      }
      anyU = umin1(acc);
      r = (s1 | anyU) & ~s0;
    }
    for (uint32_t d = 0; d < nds; ++d) {
      const int b = ext_slot((int)d);
      const uint32_t lm = rec.get(b);
      const T dMs = AR::of(rec.get(b + 1), rec.get(b + 2));
      const uint32_t x = rec.get(b + 3);
      const uint32_t i = x & 0xFFFFu, nl = x >> 16;
      uint32_t later = sc.Rwin & lm;
      for (uint32_t l = 0; l < nl; ++l) {
        const uint32_t u = node16(b + 4, l);
        later |= bit(A.at_word(u >> 5), u & 31);
      }
      later = umin1(later);
      const uint32_t fr = r & ~bit(B.at_word(i >> 5), i & 31) & ~later & 1u;
      val = AR::madd(val, fr, dMs);
    }
  } else {
    // nodes outside both formats: walk the CSR lists
    anyU = 0;
    const int ue = a.user_ptr[v + 1];
    for (int e = a.user_ptr[v]; e < ue; ++e) {
      const int u = a.user_idx[e];
      if (u > t) break;
      anyU |= r_bit(u, v, sc.Rwin, A);
    }
    r = ((s1 | anyU) & ~s0 & 1u) | (uint32_t)kFirst;
    val = AR::madd(val, r & ~s1 & ~anyU & 1u, Mv);
    const int de = a.dep_ptr[v + 1];
    for (int e = a.dep_ptr[v]; e < de; ++e) {
      const int i = a.dep_idx[e];
      uint32_t later = 0;
      const int le = a.user_ptr[i + 1];
      for (int e2 = a.dep_upos[e]; e2 < le; ++e2) {
        const int u = a.user_idx[e2];
        if (u > t) break;
        later |= r_bit(u, v, sc.Rwin, A);
      }
      const uint32_t fr = r & ~bit(B.word(i >> 5), i & 31) & ~later & 1u;
      val = AR::madd(val, fr, AR::of_i(a.M[i]));
    }
  }
  sc.cost = AR::madd(sc.cost, r, Cv);
  sc.U0 = AR::madd(sc.U0, s0, Mv);
  // Keep both sums here: left free, the compiler sinks them to the end of
  // the unrolled loop, which keeps a fourth record buffer alive and adds
  // register copies to every iteration.
  asm volatile("" : "+v"(sc.cost), "+v"(sc.U0));
  sc.maxv = AR::max(sc.maxv, val);
  sc.Y = AR::msub(val, r, Mv);
  // slide the window down by one node: bit 0 becomes node v
  sc.Rwin = (sc.Rwin << 1) | r;
  if (__builtin_expect(jj == 0, 0)) {  // chunk finished: R_t replaces S_t, move to the next chunk
    const int c = v >> 5;
    A.word(c) = sc.Rwin;
    if (c > 0) {
      sc.w0 = A.word(c - 1);
      sc.w1 = B.word(c - 1);
    }
  }
}

// Descriptor of the node-record array.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rec_rsrc(const EvalArgs& a) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint4*>(a.recs), 0, a.n * kNodeRecBytes, kBufWord3);
}

__device__ __forceinline__ void settle_w(uint32_t w) { asm volatile("" ::"v"(w)); }
__device__ __forceinline__ void settle_f(const RecF& f) {
  asm volatile("" ::"v"(f.mc.x), "v"(f.mc.y), "v"(f.mc.z), "v"(f.mc.w), "v"(f.dm.x), "v"(f.dm.y), "v"(f.dm.z),
               "v"(f.dm.w));
}

// Pipeline shape per row storage: with S_{t+1} in 32 registers (n < 1024)
// the kernel runs 5 waves per SIMD if it stays within 96 VGPRs, so the fp64
// record group comes one node ahead (two buffers) and only dependency slots
// 0-1 are pipelined; the wider variants run 1-2 waves per SIMD, where
// latency matters more than registers: the fp64 group two nodes ahead (four
// buffers) and all four slots pipelined.
template <typename RowB> struct PipeShape { static constexpr int kFAhead = 2, kSlots = 4; };
template <> struct PipeShape<RowReg> { static constexpr int kFAhead = 1, kSlots = 2; };

// One node of the scan, software-pipelined: the record dword of node v - 2
// and the fp64 record group of node v - kFAhead are requested, the LDS words
// of node v - 1 are requested, then node v is evaluated. Record dwords and
// fp64 groups rotate through four buffers (two for the groups one node
// ahead), LDS words through two, so registers never move within a turn of
// the 4-node unrolled loop.
template <bool kWide, int CW, bool kFirst, typename RowB>
__device__ __forceinline__ void pipe_step(const EvalArgs& a, int t, int v, uint32_t (&rw)[4], RecF (&rf)[4],
                                          LdsVals<PipeShape<RowB>::kSlots> (&lb)[2],
                                          Scan<typename Ar<kWide>::T>& sc, Row A, RowB& B) {
  constexpr int kFA = PipeShape<RowB>::kFAhead;
  constexpr int NW = (CW + 1) & 3, FW = (CW + 2) & 3;
  constexpr int CF = kFA == 1 ? (CW & 1) : CW;
  constexpr int LF = kFA == 1 ? (CF ^ 1) : ((CW + 2) & 3);
  constexpr int LC = CW & 1, LN = LC ^ 1;
  load_rec_w(rw[FW], rec_rsrc(a), max(v - 2, 0));
  load_rec_f(rf[LF], rec_rsrc(a), max(v - kFA, 0));
  issue_reads(rw[NW], A, B, lb[LN]);
  asm volatile("" ::: "memory");  // keep the requests ahead of this node's work
  RecRegs rec;
  rec.w = rw[CW];
  rec.mc = rf[CF].mc;
  rec.dm = rf[CF].dm;
  scan_node<kWide, kFirst>(a, t, v, rec, lb[LC], sc, A, B);
}

// One stage t of one candidate (per lane): S_t in A, S_{t+1} in B on entry,
// R_t in A on exit.
template <bool kWide, typename RowB>
__device__ __forceinline__ void eval_stage(const EvalArgs& a, int t, Row A, RowB& B, typename Ar<kWide>::T& stage_peak,
                                           typename Ar<kWide>::T& stage_cost) {
  using AR = Ar<kWide>;
  constexpr int kFA = PipeShape<RowB>::kFAhead;
  Scan<typename AR::T> sc;
  sc.U0 = AR::of_i(a.base);
  sc.Y = 0;
  sc.maxv = AR::lowest();
  sc.cost = 0;
  sc.Rwin = 0;
  sc.w0 = A.word(t >> 5);
  sc.w1 = B.word(t >> 5);
  uint32_t rw[4];
  RecF rf[4];
  LdsVals<PipeShape<RowB>::kSlots> lb[2];
  load_rec_w(rw[0], rec_rsrc(a), t);
  load_rec_w(rw[1], rec_rsrc(a), max(t - 1, 0));
  load_rec_f(rf[0], rec_rsrc(a), t);
  if (kFA == 2) load_rec_f(rf[1], rec_rsrc(a), max(t - 1, 0));
  issue_reads(rw[0], A, B, lb[0]);
  int v = t;
  pipe_step<kWide, 0, true>(a, t, v, rw, rf, lb, sc, A, B);
  const int groups = __builtin_amdgcn_readfirstlane(t / 4);
  for (int g = 0; g < groups; ++g) {
    pipe_step<kWide, 1, false>(a, t, --v, rw, rf, lb, sc, A, B);
    pipe_step<kWide, 2, false>(a, t, --v, rw, rf, lb, sc, A, B);
    pipe_step<kWide, 3, false>(a, t, --v, rw, rf, lb, sc, A, B);
    pipe_step<kWide, 0, false>(a, t, --v, rw, rf, lb, sc, A, B);
  }
  if (v >= 1) pipe_step<kWide, 1, false>(a, t, --v, rw, rf, lb, sc, A, B);
  if (v >= 1) pipe_step<kWide, 2, false>(a, t, --v, rw, rf, lb, sc, A, B);
  if (v >= 1) pipe_step<kWide, 3, false>(a, t, --v, rw, rf, lb, sc, A, B);
  // prefetches past node 0 are never read: retire them inside the stage
  settle_w(rw[0]);
  settle_w(rw[1]);
  settle_w(rw[2]);
  settle_w(rw[3]);
  settle_f(rf[0]);
  settle_f(rf[1]);
  if (kFA == 2) {
    settle_f(rf[2]);
    settle_f(rf[3]);
  }
  stage_peak = AR::stage_peak(sc.U0, sc.Y, sc.maxv);
  stage_cost = sc.cost;
}

// After stage t: S_{t+1} becomes the next stage's S_t. With S_{t+1} in
// registers it is copied into the LDS row (its words end at (t+1)/32; the LDS
// row is zero above that); with both rows in LDS they swap roles.
__device__ __forceinline__ void next_stage(Row& A, Row& B, int) {
  const Row tmp = A;
  A = B;
  B = tmp;
}
__device__ __forceinline__ void next_stage(Row& A, RowReg& B, int t) {
  const int last = (t + 1) >> 5;
#pragma unroll
  for (int w = 0; w < kRegRowWords; ++w)
    if (w <= last) A.word(w) = B.w[w];
}
template <int kVecs>
__device__ __forceinline__ void next_stage(Row& A, RowRegV<kVecs>& B, int t) {
  const int last = (t + 1) >> 5;
#pragma unroll
  for (int r = 0; r < 32; ++r) {
    if (r <= last) A.word(r) = B.v0[r];
    if (32 + r <= last) A.word(32 + r) = B.v1[r];
    if (kVecs == 4) {
      if (64 + r <= last) A.word(64 + r) = B.v2[r];
      if (96 + r <= last) A.word(96 + r) = B.v3[r];
    }
  }
}

// The stages t0 .. t1-1 of one work item: fold each stage's peak and cost.
template <bool kWide, int kSrc, typename RowB>
__device__ __forceinline__ void run_item(const EvalArgs& a, int t0, int t1, uint32_t k, bool det_lane, uint32_t rk,
                                         Row& A, RowB& B, typename Ar<kWide>::T& seg_peak, int64_t& seg_cost) {
  using AR = Ar<kWide>;
  if (t0 >= t1) return;
  gen_row<kSrc>(a, t0, k, det_lane, rk, A);
  for (int t = t0; t < t1; ++t) {
    gen_row<kSrc>(a, t + 1, k, det_lane, rk, B);
    typename AR::T sp, sc;
    eval_stage<kWide>(a, t, A, B, sp, sc);
    seg_peak = AR::seg_max(seg_peak, sp);
    seg_cost += AR::i64(sc);
    if (a.rrows) {  // R_t, now in A, kept for the best-candidate output
      uint32_t* dst = a.rrows + row_base(t) * (size_t)a.kpad + k;
      for (int w = 0; w <= (t >> 5); ++w) dst[(size_t)w * a.kpad] = A.word(w);
    }
    next_stage(A, B, t);
  }
}

// One wave per workgroup: 64 candidates over one work item (a range of
// stages). kRegW: 32, 64 or 128 when the S_{t+1} row lives in vector
// registers (rows of up to that many words) and is copied to the LDS row at
// the end of each stage, which halves the LDS a wave needs; 0 when both rows
// are in LDS and swap roles. kSrc: where the S rows come from (kSrcRound,
// kSrcUser, kSrcThreshold).
template <int kRegW, int kSrc, bool kWide = false>
__global__ void __launch_bounds__(kWave, kRegW == kRegRowWords ? 5 : 1)
ckm_eval_kernel(EvalArgs a) {
  using AR = Ar<kWide>;
  extern __shared__ uint32_t lds[];
  const int lane = threadIdx.x;
  const int group = blockIdx.x;
  const int item = blockIdx.y;
  const uint32_t k = (uint32_t)(group * kWave + lane);
  const bool det_lane = a.det0 && k == 0;
  // threshold rank of the lane's candidate (lanes past K take K-1's)
  const uint32_t rk = kSrc == kSrcThreshold ? a.rank[k < (uint32_t)a.K ? k : (uint32_t)a.K - 1u] : 0u;
  char* wave_lds = reinterpret_cast<char*>(lds);
  Row A{wave_lds + 4 * lane};
  // Rows start zeroed: words beyond a row's end (and node n's bit) read 0.
  for (int w = 0; w < a.row_words; ++w) A.word(w) = 0u;

  int t0, t1;
  item_range(a, item, t0, t1);
  typename AR::T seg_peak = AR::lowest();
  int64_t seg_cost = 0;
  if constexpr (kRegW == 0) {
    Row B{wave_lds + (size_t)a.row_words * 256 + 4 * lane};
    for (int w = 0; w < a.row_words; ++w) B.word(w) = 0u;
    run_item<kWide, kSrc>(a, t0, t1, k, det_lane, rk, A, B, seg_peak, seg_cost);
  } else if constexpr (kRegW == kRegRowWords) {
    RowReg B;
    B.w = (u32x32)0u;
    run_item<kWide, kSrc>(a, t0, t1, k, det_lane, rk, A, B, seg_peak, seg_cost);
  } else {
    u32x32 b0 = (u32x32)0u, b1 = (u32x32)0u, b2 = (u32x32)0u, b3 = (u32x32)0u;
    RowRegV<kRegW / 32> B{b0, b1, b2, b3};
    run_item<kWide, kSrc>(a, t0, t1, k, det_lane, rk, A, B, seg_peak, seg_cost);
  }
  // fold the item's result into the candidate's totals: max of the stage
  // peaks, sum of the stage costs (exact integers, any order)
  if ((int)k < a.K && t0 < t1) {
    atomicMax(reinterpret_cast<long long*>(a.part_peak) + k, (long long)AR::i64(seg_peak));
    atomicAdd(reinterpret_cast<unsigned long long*>(a.part_cost) + k, (unsigned long long)seg_cost);
  }
  if (group == 0 && item == 0 && lane == 0) a.hdr[0] = a.items;
}

// Empty totals before an evaluate launch: peak = INT64_MIN, cost = 0.
__global__ void __launch_bounds__(256) ckm_eval_init_kernel(int32_t K, int64_t* __restrict__ peak,
                                                            int64_t* __restrict__ cost) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k < K) {
    peak[k] = INT64_MIN;
    cost[k] = 0;
  }
}

// The same for the 64 candidates of one group, done by the mask producers'
// blocks of y = 0 in place of a launch of its own (peak NULL: nothing).
struct Totals {
  int64_t* __restrict__ peak;
  int64_t* __restrict__ cost;
  int32_t K;
};
__device__ __forceinline__ void clear_totals(const Totals& tot, int group) {
  const int k = group * kWave + (int)threadIdx.x;
  if (tot.peak && blockIdx.y == 0 && k < tot.K) {
    tot.peak[k] = INT64_MIN;
    tot.cost[k] = 0;
  }
}

// ---------------------------------------------------------------------------
// Thresholds: one block per row r; q[r][i] = floor(clamp(S*, 0, 1) * 2^16) for
// i < r (Section 5.1), the deterministic bits 1[S* > 0.5] of Algorithm 2, and
// a per-row NaN flag.
__global__ void __launch_bounds__(256) ckm_quantize_kernel(const double* __restrict__ s, int64_t ld,
                                                           int32_t n, int32_t ldq, int32_t det_words,
                                                           uint32_t* __restrict__ q,
                                                           uint32_t* __restrict__ det,
                                                           int32_t* __restrict__ nan_row) {
  __shared__ int any_nan;
  const int r = blockIdx.x;
  if (r >= n) return;   // the grid has one block per row
  if (threadIdx.x == 0) any_nan = 0;
  __syncthreads();
  int my_nan = 0;
  for (int i0 = 0; i0 < ldq; i0 += blockDim.x) {
    const int i = i0 + threadIdx.x;   // ldq is a multiple of 64: whole waves stay in the row
    double x = 0.0;
    const bool in = i < r;
    if (in) x = s[(int64_t)r * ld + i];
    const bool isnan_x = in && (x != x);
    my_nan |= isnan_x;
    uint32_t qv = 0;
    if (in && !isnan_x) qv = (uint32_t)floor(fmin(fmax(x, 0.0), 1.0) * 65536.0);
    if (i < ldq) q[(size_t)r * ldq + i] = qv;
    const uint64_t bits = __ballot(in && x > 0.5);
    const int lane = threadIdx.x & 63;
    if (i < ldq && (lane == 0 || lane == 32))
      det[(size_t)r * det_words + (i >> 5)] = (uint32_t)(bits >> lane);
  }
  if (my_nan) atomicOr(&any_nan, 1);
  __syncthreads();
  if (threadIdx.x == 0) nan_row[r] = any_nan;
}

// ---------------------------------------------------------------------------
// Threshold family, ranks: thread per candidate k; rank[k] = #{j : p_j < p_k}
// and p_k stored at position rank[k] + #{j < k : p_j == p_k} of the sorted
// copy (a stable counting sort; K is at most CKM_MAX_THRESHOLDS). The
// thresholds are staged through LDS in tiles of the block size.
__global__ void __launch_bounds__(256) ckm_threshold_rank_kernel(int32_t K, const double* __restrict__ p,
                                                                 double* __restrict__ sorted,
                                                                 uint32_t* __restrict__ rank) {
  __shared__ double tile[256];
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  const double pk = k < K ? p[k] : 0.0;
  uint32_t lt = 0, eq = 0;
  for (int j0 = 0; j0 < K; j0 += 256) {
    __syncthreads();
    if (j0 + (int)threadIdx.x < K) tile[threadIdx.x] = p[j0 + threadIdx.x];
    __syncthreads();
    const int m = min(256, K - j0);
    for (int jj = 0; jj < m; ++jj) {
      const double pj = tile[jj];
      lt += pj < pk ? 1u : 0u;
      eq += (pj == pk && j0 + jj < k) ? 1u : 0u;
    }
  }
  if (k < K) {
    rank[k] = lt;
    sorted[lt + eq] = pk;   // lt + eq <= K - 1: both count distinct j != k
  }
}

// Threshold family, keys: one block per row r; q[r][i] = #{j : p_j <
// clamp(S*[r][i], 0, 1)} for i < r (a lower-bound search of the sorted
// thresholds), 0 elsewhere. The row's NaN flag covers S*; row 0, which has
// no entries, carries the flag for NaN thresholds.
__global__ void __launch_bounds__(256) ckm_threshold_key_kernel(const double* __restrict__ s, int64_t ld,
                                                                int32_t n, int32_t ldq, int32_t K,
                                                                const double* __restrict__ p,
                                                                const double* __restrict__ sorted,
                                                                uint32_t* __restrict__ q,
                                                                int32_t* __restrict__ nan_row) {
  __shared__ int any_nan;
  const int r = blockIdx.x;
  if (r >= n) return;   // the grid has one block per row
  if (threadIdx.x == 0) any_nan = 0;
  __syncthreads();
  int my_nan = 0;
  if (r == 0)
    for (int k = threadIdx.x; k < K; k += blockDim.x) my_nan |= p[k] != p[k];
  for (int i0 = 0; i0 < ldq; i0 += blockDim.x) {
    const int i = i0 + threadIdx.x;
    const bool in = i < r;
    double x = in ? s[(int64_t)r * ld + i] : 0.0;
    const bool isnan_x = in && (x != x);
    my_nan |= isnan_x;
    uint32_t key = 0;
    if (in && !isnan_x) {
      x = fmin(fmax(x, 0.0), 1.0);
      // first position whose threshold is not below x
      uint32_t lo = 0, len = (uint32_t)K;
      while (len > 0) {
        const uint32_t half = len >> 1;
        if (sorted[lo + half] < x) {
          lo += half + 1;
          len -= half + 1;
        } else {
          len = half;
        }
      }
      key = lo;
    }
    if (i < ldq) q[(size_t)r * ldq + i] = key;
  }
  if (my_nan) atomicOr(&any_nan, 1);
  __syncthreads();
  if (threadIdx.x == 0) nan_row[r] = any_nan;
}

// ---------------------------------------------------------------------------
// Per-candidate feasibility and the block's lexicographic minimum of
// (cost, peak, k) over feasible candidates.
struct Best {
  int64_t cost, peak;
  int32_t k, pad;
};

__device__ __forceinline__ bool better(const Best& x, const Best& y) {
  if (x.k < 0) return false;
  if (y.k < 0) return true;
  if (x.cost != y.cost) return x.cost < y.cost;
  if (x.peak != y.peak) return x.peak < y.peak;
  return x.k < y.k;
}

// One thread per candidate: copy out its totals, test the budget, then the
// block's minimum.
__global__ void __launch_bounds__(256) ckm_reduce_kernel(int32_t K, const int64_t* __restrict__ tot_peak,
                                                         const int64_t* __restrict__ tot_cost,
                                                         int64_t budget, int64_t* __restrict__ peak,
                                                         int64_t* __restrict__ cost,
                                                         uint8_t* __restrict__ feasible,
                                                         Best* __restrict__ block_best) {
  __shared__ Best sb[256];
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  Best b{0, 0, -1, 0};
  if (k < K) {
    const int64_t p = tot_peak[k], c = tot_cost[k];
    peak[k] = p;
    cost[k] = c;
    const bool f = p <= budget;
    feasible[k] = f ? 1 : 0;
    if (f) b = Best{c, p, k, 0};
  }
  sb[threadIdx.x] = b;
  __syncthreads();
  for (int off = blockDim.x / 2; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off && better(sb[threadIdx.x + off], sb[threadIdx.x]))
      sb[threadIdx.x] = sb[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) block_best[blockIdx.x] = sb[0];
}

__global__ void __launch_bounds__(256) ckm_argmin_kernel(int32_t nblocks, const Best* __restrict__ block_best,
                                                         int32_t n, const int32_t* __restrict__ nan_row,
                                                         int32_t* __restrict__ best_k,
                                                         int32_t* __restrict__ status) {
  __shared__ Best sb[256];
  __shared__ int any_nan;
  if (threadIdx.x == 0) any_nan = 0;
  Best b{0, 0, -1, 0};
  for (int i = threadIdx.x; i < nblocks; i += blockDim.x)
    if (better(block_best[i], b)) b = block_best[i];
  int nan = 0;
  for (int r = threadIdx.x; r < n; r += blockDim.x) nan |= nan_row[r];
  sb[threadIdx.x] = b;
  __syncthreads();
  if (nan) atomicOr(&any_nan, 1);
  for (int off = blockDim.x / 2; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off && better(sb[threadIdx.x + off], sb[threadIdx.x]))
      sb[threadIdx.x] = sb[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    best_k[0] = sb[0].k;
    if (status) status[0] = any_nan ? (int32_t)CKM_E_INVALID_ARG : (int32_t)CKM_OK;
  }
}

// Both steps in one block of 1024 threads, for K up to kSelectOneBlock: each
// thread walks candidates tid, tid + 1024, ... (in increasing k, so among
// equal (cost, peak) it keeps the smallest k), then the block's minimum.
constexpr int kSelectOneBlock = 1 << 16;
__global__ void __launch_bounds__(1024) ckm_select_kernel(int32_t K, const int64_t* __restrict__ tot_peak,
                                                          const int64_t* __restrict__ tot_cost, int64_t budget,
                                                          int64_t* __restrict__ peak, int64_t* __restrict__ cost,
                                                          uint8_t* __restrict__ feasible, int32_t n,
                                                          const int32_t* __restrict__ nan_row,
                                                          int32_t* __restrict__ best_k,
                                                          int32_t* __restrict__ status) {
  __shared__ Best sb[1024];
  __shared__ int any_nan;
  if (threadIdx.x == 0) any_nan = 0;
  Best b{0, 0, -1, 0};
  for (int k = threadIdx.x; k < K; k += blockDim.x) {
    const int64_t p = tot_peak[k], c = tot_cost[k];
    peak[k] = p;
    cost[k] = c;
    const bool f = p <= budget;
    feasible[k] = f ? 1 : 0;
    const Best x{c, p, k, 0};
    if (f && better(x, b)) b = x;
  }
  int nan = 0;
  for (int r = threadIdx.x; r < n; r += blockDim.x) nan |= nan_row[r];
  sb[threadIdx.x] = b;
  __syncthreads();
  if (nan) atomicOr(&any_nan, 1);
  for (int off = blockDim.x / 2; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off && better(sb[threadIdx.x + off], sb[threadIdx.x]))
      sb[threadIdx.x] = sb[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    best_k[0] = sb[0].k;
    if (status) status[0] = any_nan ? (int32_t)CKM_E_INVALID_ARG : (int32_t)CKM_OK;
  }
}

// ---------------------------------------------------------------------------
// Largest batch multiplier per candidate (the maximum-batch experiment of
// the evaluation): with node sizes B * M_i (M_in, M_param fixed) every U term
// but the constant base = M_in + 2 M_param scales with B, so the peak at B is
// base + B (peak - base) and the largest B within the budget is
// floor((budget - base) / (peak - base)). Candidates over the cost cap (eq.
// cost_constr) or over the budget at B = 1 get 0; a candidate with no
// activation bytes gets INT64_MAX. The best: largest B, then the
// lexicographic minimum of (cost, peak, k); k = -1 when every B is 0.
struct BestB {
  int64_t B, cost, peak;
  int32_t k, pad;
};

__device__ __forceinline__ bool better_b(const BestB& x, const BestB& y) {
  if (x.k < 0) return false;
  if (y.k < 0) return true;
  if (x.B != y.B) return x.B > y.B;
  if (x.cost != y.cost) return x.cost < y.cost;
  if (x.peak != y.peak) return x.peak < y.peak;
  return x.k < y.k;
}

__global__ void __launch_bounds__(256) ckm_batch_kernel(int32_t K, const int64_t* __restrict__ tot_peak,
                                                        const int64_t* __restrict__ tot_cost, int64_t base,
                                                        int64_t budget, int64_t cost_cap,
                                                        int64_t* __restrict__ batch, BestB* __restrict__ block_best) {
  __shared__ BestB sb[256];
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  BestB b{0, 0, 0, -1, 0};
  if (k < K) {
    const int64_t p = tot_peak[k], c = tot_cost[k];
    int64_t B = 0;
    if (c <= cost_cap && p <= budget) B = p > base ? (budget - base) / (p - base) : INT64_MAX;
    batch[k] = B;
    if (B > 0) b = BestB{B, c, p, k, 0};
  }
  sb[threadIdx.x] = b;
  __syncthreads();
  for (int off = blockDim.x / 2; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off && better_b(sb[threadIdx.x + off], sb[threadIdx.x])) sb[threadIdx.x] = sb[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) block_best[blockIdx.x] = sb[0];
}

__global__ void __launch_bounds__(256) ckm_batch_argmax_kernel(int32_t nblocks, const BestB* __restrict__ block_best,
                                                               int32_t n, const int32_t* __restrict__ nan_row,
                                                               int32_t* __restrict__ best_k,
                                                               int64_t* __restrict__ best_batch,
                                                               int32_t* __restrict__ status) {
  __shared__ BestB sb[256];
  __shared__ int any_nan;
  if (threadIdx.x == 0) any_nan = 0;
  BestB b{0, 0, 0, -1, 0};
  for (int i = threadIdx.x; i < nblocks; i += blockDim.x)
    if (better_b(block_best[i], b)) b = block_best[i];
  int nan = 0;
  for (int r = threadIdx.x; r < n; r += blockDim.x) nan |= nan_row[r];
  sb[threadIdx.x] = b;
  __syncthreads();
  if (nan) atomicOr(&any_nan, 1);
  for (int off = blockDim.x / 2; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off && better_b(sb[threadIdx.x + off], sb[threadIdx.x])) sb[threadIdx.x] = sb[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    best_k[0] = sb[0].k;
    if (best_batch) best_batch[0] = sb[0].k >= 0 ? sb[0].B : 0;
    if (status) status[0] = any_nan ? (int32_t)CKM_E_INVALID_ARG : (int32_t)CKM_OK;
  }
}

// ---------------------------------------------------------------------------
// Best candidate's S rows: thread per (row r, 32-bit word w). Output rows
// have row_words words; words with no node (32w >= n) are zero. rank: the
// threshold family (q holds keys), else randomized or deterministic rounding.
// With R_rows, the same threads also gather the best candidate's R rows
// from the R rows the evaluate kernel kept (words above r/32 are zero).
__global__ void __launch_bounds__(256) ckm_best_rows_kernel(const uint32_t* __restrict__ q,
                                                            const uint32_t* __restrict__ det,
                                                            int32_t n, int32_t ldq, int32_t det_words,
                                                            int32_t row_words, uint32_t key0,
                                                            uint32_t key1, uint32_t det0,
                                                            const uint32_t* __restrict__ rank,
                                                            const int32_t* __restrict__ best_k,
                                                            uint32_t* __restrict__ S_rows,
                                                            const uint32_t* __restrict__ rrows, int32_t kpad,
                                                            uint32_t* __restrict__ R_rows) {
  const int r = blockIdx.y;
  const int w = blockIdx.x * blockDim.x + threadIdx.x;
  if (w >= row_words) return;
  const int bk = best_k[0];
  if (R_rows) {
    uint32_t rw = 0;
    if (bk >= 0 && w <= (r >> 5)) rw = rrows[(row_base(r) + w) * (size_t)kpad + bk];
    R_rows[(size_t)r * row_words + w] = rw;
  }
  uint32_t word = 0;
  if (bk >= 0 && 32 * w < n) {
    if (rank)
      word = threshold_word<false>(q + (size_t)r * ldq, w, r, rank[bk]);
    else if (det0 && bk == 0)
      word = det[(size_t)r * det_words + w];
    else
      word = round_word<false>(q + (size_t)r * ldq, w, r, (uint32_t)bk, key0, key1);
  }
  S_rows[(size_t)r * row_words + w] = word;
}

// Best candidate's R rows from the R rows the evaluate stage kept for every
// candidate: thread per (row t, 32-bit word w). Words above t/32 (no node
// at or below t), and every word when nothing is feasible, are zero.
__global__ void __launch_bounds__(256) ckm_best_rrows_kernel(const uint32_t* __restrict__ rrows, int32_t kpad,
                                                             int32_t row_words,
                                                             const int32_t* __restrict__ best_k,
                                                             uint32_t* __restrict__ R_rows) {
  const int t = blockIdx.y;
  const int w = blockIdx.x * blockDim.x + threadIdx.x;
  if (w >= row_words) return;
  const int bk = best_k[0];
  uint32_t word = 0;
  if (bk >= 0 && w <= (t >> 5)) word = rrows[(row_base(t) + w) * (size_t)kpad + bk];
  R_rows[(size_t)t * row_words + w] = word;
}

// Best candidate's R rows: lane = stage t (64 stages per wave), Algorithm
// 2's right-to-left repair over nodes v = (last stage of the wave) .. 0, all
// lanes at the same node. As in the evaluate kernel, the R bits of the 32
// nodes above v sit in a one-register window and R words of finished chunks
// sit in an LDS row per lane ([word][lane]) for users beyond the window. With
// one wave per SIMD nothing hides latency, so node records come 32 at a time
// (a chunk, one register each, lane L holding dword L) one chunk ahead, and
// the lane's S_t and S_{t+1} rows are copied to LDS first. A lane whose stage
// is below v computes nothing there. Bits of the S rows on or above the
// diagonal are never decisive: node t is computed whatever S_t[t] holds.
// Dynamic LDS: three rows (R, S_t, S_{t+1}) of n / 32 + 1 words per lane.
struct ClosureArgs {
  int32_t n, row_words;
  const int32_t* user_ptr;
  const int32_t* user_idx;
  const uint4* recs;
  const int32_t* best_k;
  const uint32_t* S_base;
  size_t cand_stride;
  uint32_t* R_rows;
};

constexpr int kChunk = 32;

// Records of nodes 32c .. 32c + 31 (clamped to node n - 1), lane L holding
// dword L of each.
__device__ __forceinline__ void load_chunk(uint32_t (&rec)[kChunk], const uint4* recs, int c, int n) {
  const size_t lane_off = (size_t)((threadIdx.x & 63u) * 4u);
#pragma unroll
  for (int j = 0; j < kChunk; ++j) {
    const int v = __builtin_amdgcn_readfirstlane(min(kChunk * c + j, n - 1));
    rec[j] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const char*>(recs) + (size_t)v * kNodeRecBytes +
                                                 lane_off);
  }
}

__device__ __forceinline__ uint32_t rl(uint32_t w, int i) { return __builtin_amdgcn_readlane(w, i); }

// Nodes 32c + 31 .. 32c of the scan for the lane's stage t.
__device__ __forceinline__ void closure_chunk(const ClosureArgs& a, int c, int t, int tmax, const uint32_t (&rec)[kChunk],
                                              Row A, Row S0, Row S1, uint32_t& Rwin) {
  const uint32_t w0 = S0.word(c), w1 = S1.word(c);
  uint32_t far_next = A.at_word(word_at(rl(rec[kChunk - 1], kDwRefs0), 0));
#pragma unroll
  for (int jj = kChunk - 1; jj >= 0; --jj) {
    const int v = kChunk * c + jj;
    const uint32_t far_w = far_next;
    if (jj > 0) far_next = A.at_word(word_at(rl(rec[jj - 1], kDwRefs0), 0));
    uint32_t r = 0;
    if (v <= tmax) {
      const uint32_t um = rl(rec[jj], kDwUmask), b0 = rl(rec[jj], kDwBits0);
      pin_s(um, b0, b0);
      bool slow = false;
      if (__builtin_expect((b0 >> 30) == 3u, 0)) slow = (rl(rec[jj], kDwRefs1) & kRefsSlow) != 0u;
      uint32_t anyU;
      if (__builtin_expect(!slow, 1)) {
        anyU = umin1(and_or(Rwin, um, __builtin_amdgcn_ubfe(far_w, b0, 1)));
      } else {
        // more than one user beyond the window: walk the users
        anyU = 0;
        const int ue = a.user_ptr[v + 1];
        for (int e = a.user_ptr[v]; e < ue; ++e) {
          const int u = a.user_idx[e];
          const int d = u - v - 1;
          anyU |= d < 32 ? bit(Rwin, d) : bit(A.word(u >> 5), u & 31);
        }
      }
      r = ((bit(w1, jj) | anyU) & ~bit(w0, jj)) & 1u;
      if (v == t) r = 1u;
      if (v > t) r = 0u;
    }
    Rwin = (Rwin << 1) | r;
  }
  A.word(c) = Rwin;
}

__global__ void __launch_bounds__(kWave) ckm_best_closure_kernel(ClosureArgs a) {
  extern __shared__ uint32_t lds_c[];
  const int lane = threadIdx.x;
  const int t = blockIdx.x * kWave + lane;
  const bool active = t < a.n;
  const int tmax = min(a.n - 1, (int)blockIdx.x * kWave + kWave - 1);
  const int bk = a.best_k[0];
  uint32_t* Rout = a.R_rows + (size_t)(active ? t : 0) * a.row_words;
  if (bk < 0) {
    if (active)
      for (int w = 0; w < a.row_words; ++w) Rout[w] = 0u;
    return;
  }
  const int lwords = (a.n >> 5) + 1;
  char* base = reinterpret_cast<char*>(lds_c) + 4 * lane;
  Row A{base}, S0{base + (size_t)lwords * 256}, S1{base + (size_t)2 * lwords * 256};
  // the lane's rows; words past its stage read as zero (never decisive)
  const int ts = active ? t : tmax;
  const uint32_t* src0 = a.S_base + (size_t)bk * a.cand_stride + (size_t)ts * a.row_words;
  const uint32_t* src1 = src0 + a.row_words;
  const bool has1 = ts + 1 < a.n;
  for (int w = 0; w < lwords; ++w) {
    const bool in = w <= (ts >> 5);
    A.word(w) = 0u;
    S0.word(w) = in ? src0[w] : 0u;
    S1.word(w) = (in && has1) ? src1[w] : 0u;
  }
  uint32_t Rwin = 0;
  uint32_t ra[kChunk], rb[kChunk];
  int c = tmax >> 5;
  load_chunk(ra, a.recs, c, a.n);
  for (;;) {
    if (c >= 1) load_chunk(rb, a.recs, c - 1, a.n);
    closure_chunk(a, c, t, tmax, ra, A, S0, S1, Rwin);
    if (--c < 0) break;
    if (c >= 1) load_chunk(ra, a.recs, c - 1, a.n);
    closure_chunk(a, c, t, tmax, rb, A, S0, S1, Rwin);
    if (--c < 0) break;
  }
  if (active)
    for (int w = 0; w < a.row_words; ++w) Rout[w] = w <= (t >> 5) ? A.word(w) : 0u;
}

// ---------------------------------------------------------------------------
// Mask path. A group's 64 candidates share one 64-bit word per (stage row,
// node): bit j is candidate 64g + j. With the rows in that form, the repair
// of Algorithm 2 and the FREE tests of eq. collectable become scalar-unit
// operations on whole words (one instruction decides a node for all 64
// candidates), and the vector unit keeps only the sums, each a masked
// binary64 update selected by such a word. A node's record and its S words
// come through the scalar cache; the R bits of the nodes above it stay in
// each lane's window register and register row, as in the kernel above.
//
// Mask rows of a group: row t holds 8 (t/8 + 1) words (nodes 0 .. t rounded
// up to whole blocks of 8; words for nodes >= t are zero); row n, after the
// last stage, is all zero.
__host__ __device__ __forceinline__ size_t mrow_off(int t) {
  const size_t q = (size_t)(t >> 3), r = (size_t)(t & 7);
  return 8 * ((size_t)t + 4 * q * (q ? q - 1 : 0) + q * r);
}

// Node v's data, 128 bytes at 128 v:
//   [0, 64)   record, 16 dwords (one scalar load)
//   [64, 96)  slots 2-3 (nodes with three or four dependencies): lm, ref of
//             slot 2, of slot 3, dependency count, byte offsets in a mask
//             row of the S_{t+1} words of the slot 2 and 3 dependencies
//   [96, 112) binary64 M of slots 2 and 3
// A far reference names a node u more than 32 above v as u << 16 | (u & 31)
// (none: 0xFFFF << 16). Its R bit matters only when u <= t, i.e. when the
// field is below (t + 1) << 16: a node above t computes nothing in stage t.
// Record words:
//   0: users u of v with u <= v + 32 (bit u - v - 1)
//   1: ctrl: far reference to the user of v more than 32 above it | slots
//      2-3 present << 8
//   slot s (words 2 + 2s, 3 + 2s):
//      lm: users u of the dependency with v < u <= v + 32 (bit u - v - 1)
//      ref: far reference to the dependency's later user
//      An absent slot has lm = 0 and no far reference: it frees nothing, its
//      size being 0.
//   6: for node v-1, the byte offset in a mask row of the S_{t+1} word of
//      its slot 0 dependency (0 for an absent slot), fetched one node ahead
//   7: high half: the gate, the high half of the least of the node's three
//      far references (words 1, 3 and 5), or 0 when the node has more than
//      two dependencies: when the word is at or above the stage's limit
//      (t + 1) << 16, the node is decided in a form without far lookups or
//      rare slots (the limit's low half is 0, so the low half of the word
//      never decides). Low half: for node v-1, the byte offset of its slot 1
//      dependency's S_{t+1} word, as word 6. (Both offsets in word 6 cost a
//      shift and a mask per node.)
//   8-15: binary64 M_v, C_v, M of slots 0 and 1, used from scalar registers
//      (the vector registers they would take are worth a wave per SIMD)
// Pairs of nodes are aligned (nodes 2c, 2c+1). A stage's scan starts at the
// top of its node's pair; a node above t there (or past n - 1, whose data is
// padded with empty nodes up to np = round_up(n, 4) + 4) computes nothing
// and holds nothing, so it leaves every sum unchanged.
constexpr uint32_t kMNoFar = 0xFFFFu << 16, kMRare = 1u << 8;
constexpr int kMNodeBytes = 128;
__host__ __device__ __forceinline__ int mask_padded_nodes(int n) { return ((n + 3) & ~3) + 4; }

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x16 __attribute__((ext_vector_type(16)));

struct MaskArgs {
  int32_t n, K, items, kind, P, T0, R1, R2;   // work plan (see Plan)
  int32_t np;                                 // padded node count of the node data
  double base;                                // M_in + 2 M_param
  size_t mgroup;                              // words of one group's mask rows
  cptr<uint64_t> mrows;                       // S masks, group-major
  cptr<u32x16> mnodes;                        // np x 128 bytes of node data
  uint32_t* __restrict__ rrows;               // R rows out (row array layout), or NULL
  int32_t kpad;
  int64_t* __restrict__ part_peak;
  int64_t* __restrict__ part_cost;
  int32_t* __restrict__ hdr;
  int32_t g0;                                 // group of blockIdx.x = 0
};

__device__ __forceinline__ bool lane_of(uint64_t m) { return __builtin_amdgcn_inverse_ballot_w64(m); }
__device__ __forceinline__ uint64_t mask_of(bool b) { return __builtin_amdgcn_ballot_w64(b); }
// acc + [lane's bit of m] * x, one masked binary64 update
__device__ __forceinline__ double madd_m(double acc, uint64_t m, double x) {
  return fma(lane_of(m) ? 1.0 : 0.0, x, acc);
}
// A scalar load at a 32-bit byte offset from a base (one instruction, the
// offset in a register).
template <typename T, typename B>
__device__ __forceinline__ T sload(cptr<B> base, uint32_t off) {
  return *(const __attribute__((address_space(4))) T*)((const __attribute__((address_space(4))) char*)base + off);
}
// 16 bytes at byte offset off + kOff of the node data, in every lane
template <int kOff>
__device__ __forceinline__ uint4 load_mval(__amdgpu_buffer_rsrc_t rs, uint32_t off) {
  const auto x = __builtin_amdgcn_raw_buffer_load_b128(rs, kOff, (int)off, 0);
  return make_uint4(x[0], x[1], x[2], x[3]);
}

struct MScan {
  double U0, Y, maxv, cost;
  uint32_t Rwin;   // R bits of nodes v+1 .. v+32 (bit d <-> node v + 1 + d)
};

// The R bit of the far node that field f names (more than 32 above the node
// being decided: its word of the register row is complete). A shift uses the
// low five bits of its count by itself. Only for u <= t; the empty asm keeps
// the compiler from hoisting the indexed register read out of that branch
// (the word index is clamped to the row all the same).
__device__ __forceinline__ uint32_t far_bit(const u32x32& Rrow, uint32_t f) {
  asm volatile("");
  return (Rrow[(f >> 21) & 31u] >> (f & 31u)) & 1u;
}

// One dependency slot of node v: the dependency's value is released after
// v (FREE(t,i,v) = 1) on the candidates that compute v, do not keep the
// value into stage t+1 and compute none of its later users in stage t.
template <bool kFar>
__device__ __forceinline__ double mask_slot(double val, uint64_t R, uint32_t lm, uint32_t ref, double Mi,
                                            uint64_t s1i, uint32_t Rwin, const u32x32& Rrow, uint32_t tlim) {
  uint32_t y = Rwin & lm;
  if (kFar && __builtin_expect(ref < tlim, 0)) y |= far_bit(Rrow, ref);
  const uint64_t later = mask_of(y != 0u);
  const uint64_t fr = R & ~(s1i | later);
  return madd_m(val, fr, Mi);
}

// What node v needs besides its block: its record, the S_{t+1} words of its
// slot 0 and 1 dependencies and its binary64 operands (M_v, C_v | M of slots
// 0, 1), all requested one node ahead.
struct MNode {
  u32x16 rec;
  uint64_t d0, d1;
};

// Node v of stage t for the 64 candidates of a group: S0, S1 are the words
// of S_t[v] and S_{t+1}[v]. Algorithm 2: v is computed if it is node t
// (constraint 4a), or it is not held and is kept into t+1 (1c) or used by a
// computed node (1b). kTop: v is in the block of node t, and may be t; below
// that block, v < t and the scan has passed at least one node. Released
// right after its own compute (eq. collectable with i = v): a computed node
// that is neither kept nor used, which only node t can be.
// kSlow: the general form, for a node whose gate (record word 7: the least
// of its three far references, 0 with more than two dependencies) is below
// the stage's limit; the fast form has no far lookup and no rare slots.
template <bool kTop, bool kSlow, bool kSkip>
__device__ __forceinline__ void mask_node_as(const MaskArgs& a, int t, int v, const MNode& nd, uint64_t S0,
                                             uint64_t S1, cptr<uint64_t> s1row, MScan& sc, u32x32& Rrow,
                                             uint32_t tlim) {
  const u32x16& rec = nd.rec;
  const uint32_t ctrl = rec[1];
  const double Mv = dbl(rec[8], rec[9]), Cv = dbl(rec[10], rec[11]);
  uint32_t x = sc.Rwin & rec[0];
  if (kSlow && __builtin_expect(ctrl < tlim, 0)) x |= far_bit(Rrow, ctrl);
  const uint64_t x1 = S1 | mask_of(x != 0u);
  uint64_t R = x1 & ~S0;
  sc.U0 = madd_m(sc.U0, S0, Mv);
  // A lane that does not compute v frees nothing after it, and its val = Y
  // changes neither maxv (which already covers Y: the running value has only
  // fallen since the last computed node) nor Y. kSkip: a node that no
  // candidate of the group computes returns here. Without it such nodes take
  // the general path, which is faster for randomized rounding (19 % of the
  // visits on the transformer workload: 0.455 against 0.458 ms; the seen
  // kernel at n = 4001, K = 4096: 87.2 against 88.0 ms), while the threshold
  // family, whose groups hold neighbouring thresholds, has many more of them
  // and gains from the skip on those two graphs (0.557 against 0.570 ms and
  // 85.2 against 90.3 ms per call).
  if (kSkip && !kTop && R == 0ull) {
    sc.Rwin = sc.Rwin + sc.Rwin;
    return;
  }
  double val = sc.Y;
  if (kTop && v == t) {
    R = ~0ull;
    val = madd_m(val, ~x1, Mv);
  }
  val = mask_slot<kSlow>(val, R, rec[2], rec[3], dbl(rec[12], rec[13]), nd.d0, sc.Rwin, Rrow, tlim);
  val = mask_slot<kSlow>(val, R, rec[4], rec[5], dbl(rec[14], rec[15]), nd.d1, sc.Rwin, Rrow, tlim);
  if (kSlow && __builtin_expect((ctrl & kMRare) != 0u, 0)) {
    const uint32_t off = (uint32_t)v * kMNodeBytes;
    const u32x8 r2 = sload<u32x8>(a.mnodes, off + 64);
    const u32x4 m23 = sload<u32x4>(a.mnodes, off + 96);
    val = mask_slot<true>(val, R, r2[0], r2[1], dbl(m23[0], m23[1]), sload<uint64_t>(s1row, r2[5]), sc.Rwin, Rrow,
                          tlim);
    if (r2[4] >= 4)
      val = mask_slot<true>(val, R, r2[2], r2[3], dbl(m23[2], m23[3]), sload<uint64_t>(s1row, r2[6]), sc.Rwin,
                            Rrow, tlim);
  }
  // suffix form of the U recurrence (see scan_node): val = Y + freed_v
  sc.maxv = max_f64(sc.maxv, val);
  const bool rb = lane_of(R);
  const double sel = rb ? 1.0 : 0.0;
  sc.Y = fma(-sel, Mv, val);
  sc.cost = fma(sel, Cv, sc.cost);
  sc.Rwin = sc.Rwin + sc.Rwin + (rb ? 1u : 0u);
}

template <bool kTop, bool kSkip>
__device__ __forceinline__ void mask_node(const MaskArgs& a, int t, int v, const MNode& nd, uint64_t S0, uint64_t S1,
                                          cptr<uint64_t> s1row, MScan& sc, u32x32& Rrow) {
  const uint32_t tlim = (uint32_t)(t + 1) << 16;
  if (__builtin_expect(nd.rec[7] < tlim, 0))
    mask_node_as<kTop, true, kSkip>(a, t, v, nd, S0, S1, s1row, sc, Rrow, tlim);
  else
    mask_node_as<kTop, false, kSkip>(a, t, v, nd, S0, S1, s1row, sc, Rrow, tlim);
}

// x, made to depend on a word of a record that a wait delivers, so that the
// loads it addresses are issued after that wait: scalar loads complete out
// of order, and a wait for the record would wait for them as well.
__device__ __forceinline__ uint32_t after_record(uint32_t x, uint32_t word) {
  asm("" : "+s"(x) : "s"(word));
  return x;
}

// The loads node v-1 needs, issued while node v is decided: its record (with
// its operands) at byte off, and the dependency words node v's record lists
// for it.
__device__ __forceinline__ MNode mask_fetch(const MaskArgs& a, const u32x16& rec_v, cptr<uint64_t> s1row,
                                            uint32_t off) {
  MNode nx;
  nx.rec = sload<u32x16>(a.mnodes, off);
  nx.d0 = sload<uint64_t>(s1row, rec_v[6]);
  nx.d1 = sload<uint64_t>(s1row, rec_v[7] & 0xFFFFu);
  return nx;
}

// Node v at position P of its pair (P = v & 1), with the next node's loads
// issued first; at P = 0 they include the next pair's words, into Bn0 and
// Bn1 (the current pair is in B0, B1). The loads alternate between two
// buffers by position (node v's in buf[P], node v-1's into the other), so
// nothing moves from one to the other.
template <int P, bool kTop, bool kSkip>
__device__ __forceinline__ void mask_step(const MaskArgs& a, int t, int v, MNode (&buf)[2], const u32x4& B0,
                                          const u32x4& B1, u32x4& Bn0, u32x4& Bn1, cptr<uint64_t> s0row,
                                          cptr<uint64_t> s1row, MScan& sc, u32x32& Rrow, uint32_t* rrow_t) {
  constexpr int kCur = P, kNext = P ^ 1;
  const uint64_t S0 = (uint64_t)B0[2 * P] | (uint64_t)B0[2 * P + 1] << 32;
  const uint64_t S1 = (uint64_t)B1[2 * P] | (uint64_t)B1[2 * P + 1] << 32;
  const u32x16& rec = buf[kCur].rec;
  // node v-1's data (node 0 fetches its own again: nothing is left to load)
  buf[kNext] = mask_fetch(a, rec, s1row, after_record(v >= 1 ? (uint32_t)(v - 1) * kMNodeBytes : 0u, rec[6]));
  if (P == 0) {
    // pair c-1 (v = 2c) starts 16 (c - 1) bytes into a row (0 for c = 0)
    const uint32_t boff = after_record(v >= 2 ? 8u * (uint32_t)v - 16u : 0u, rec[6]);
    Bn0 = sload<u32x4>(s0row, boff);
    Bn1 = sload<u32x4>(s1row, boff);
  }
  // The loads stay ahead of the node's gate branch. Placed after it, in a
  // block that both forms of the node share, they made the compiler route
  // the fast form through a flag, a test and a taken jump per node pair
  // (0.456 against 0.452 ms on the transformer workload).
  asm volatile("" ::: "memory");
  mask_node<kTop, kSkip>(a, t, v, buf[kCur], S0, S1, s1row, sc, Rrow);
  if (P == 0 && (v & 31) == 0) {
    // the R bits of nodes v .. v+31 are complete: one word of R_t, kept in
    // the register row (and stored for the output)
    Rrow[v >> 5] = sc.Rwin;
    if (rrow_t) rrow_t[(size_t)(v >> 5) * a.kpad] = sc.Rwin;
  }
}

// Pair c (nodes 2c+1, 2c) from B0, B1; pair c-1 loaded into Bn0, Bn1.
template <bool kTop, bool kSkip>
__device__ __forceinline__ void mask_block(const MaskArgs& a, int t, int c, MNode (&buf)[2], const u32x4& B0,
                                           const u32x4& B1, u32x4& Bn0, u32x4& Bn1, cptr<uint64_t> s0row,
                                           cptr<uint64_t> s1row, MScan& sc, u32x32& Rrow, uint32_t* rrow_t) {
  mask_step<1, kTop, kSkip>(a, t, 2 * c + 1, buf, B0, B1, Bn0, Bn1, s0row, s1row, sc, Rrow, rrow_t);
  mask_step<0, kTop, kSkip>(a, t, 2 * c, buf, B0, B1, Bn0, Bn1, s0row, s1row, sc, Rrow, rrow_t);
}

// One wave per work item: the 64 candidates of group blockIdx.x over the
// stages of item blockIdx.y. Graphs up to 1023 nodes (R row in 32 registers),
// none of whose nodes exceed the record (at most four dependencies, one user
// more than 32 nodes above the node, one such later user per dependency).
// Each node's loads are issued one node ahead, in one batch, so that a node
// waits once, for loads that had a whole node's work to arrive.
template <bool kSkip>
__global__ void __launch_bounds__(kWave) ckm_mask_eval_kernel(MaskArgs a) {
  const int lane = threadIdx.x;
  const int group = blockIdx.x + a.g0;
  const int item = blockIdx.y;
  const uint32_t k = (uint32_t)(group * kWave + lane);
  int t0, t1;
  item_range(a, item, t0, t1);
  const cptr<uint64_t> rows = a.mrows + (size_t)group * a.mgroup;
  u32x32 Rrow = (u32x32)0u;
  double seg_peak = -INFINITY;
  int64_t seg_cost = 0;
  for (int t = t0; t < t1; ++t) {
    const cptr<uint64_t> s0row = rows + mrow_off(t);
    const cptr<uint64_t> s1row = rows + mrow_off(t + 1);
    uint32_t* rrow_t = a.rrows ? a.rrows + row_base(t) * (size_t)a.kpad + k : nullptr;
    MScan sc;
    sc.U0 = (double)a.base;
    sc.Y = 0.0;
    sc.maxv = -INFINITY;
    sc.cost = 0.0;
    sc.Rwin = 0u;
    // the scan starts at the top of t's pair: node 2c + 1, whose loads node
    // 2c + 2's record names
    const int c = t >> 1;
    MNode buf[2];
    const u32x16 top = a.mnodes[(size_t)(2 * c + 2) * (kMNodeBytes / 64)];
    buf[1] = mask_fetch(a, top, s1row, (uint32_t)(2 * c + 1) * kMNodeBytes);
    const u32x4 T0 = sload<u32x4>(s0row, 16u * c), T1 = sload<u32x4>(s1row, 16u * c);
    u32x4 A0, A1, B0, B1;
    mask_block<true, kSkip>(a, t, c, buf, T0, T1, B0, B1, s0row, s1row, sc, Rrow, rrow_t);
    int cc = c - 1;
    for (; cc >= 1; cc -= 2) {
      mask_block<false, kSkip>(a, t, cc, buf, B0, B1, A0, A1, s0row, s1row, sc, Rrow, rrow_t);
      mask_block<false, kSkip>(a, t, cc - 1, buf, A0, A1, B0, B1, s0row, s1row, sc, Rrow, rrow_t);
    }
    if (cc == 0) mask_block<false, kSkip>(a, t, 0, buf, B0, B1, A0, A1, s0row, s1row, sc, Rrow, rrow_t);
    seg_peak = fmax(seg_peak, sc.U0 - sc.Y + sc.maxv);
    seg_cost += (int64_t)sc.cost;
  }
  if ((int)k < a.K && t0 < t1) {
    atomicMax(reinterpret_cast<long long*>(a.part_peak) + k, (long long)seg_peak);
    atomicAdd(reinterpret_cast<unsigned long long*>(a.part_cost) + k, (unsigned long long)seg_cost);
  }
  if (group == 0 && item == 0 && lane == 0) a.hdr[0] = a.items;
}

}  // namespace
// v_writelane_b32 through its compiler intrinsic, so that the compiler sees
// the instruction and its hazards (this compiler has no builtin for it). The
// declaration binds a name to the intrinsic, so it stays outside the unnamed
// namespace: there it would name an internal function that is never defined.
__device__ int amdgcn_writelane(int x, int lane, int v) __asm("llvm.amdgcn.writelane.i32");
namespace {
// Lane L of v takes the wave-uniform x.
template <int L>
__device__ __forceinline__ uint32_t write_lane(uint32_t v, uint32_t x) {
  return (uint32_t)amdgcn_writelane((int)x, L, (int)v);
}
// Lanes 2j and 2j+1 take the low and high halves of m[j], j >= J.
template <int J>
__device__ __forceinline__ uint32_t put_masks(uint32_t v, const uint64_t (&m)[8]) {
  v = write_lane<2 * J>(v, (uint32_t)m[J]);
  v = write_lane<2 * J + 1>(v, (uint32_t)(m[J] >> 32));
  if constexpr (J + 1 < 8) v = put_masks<J + 1>(v, m);
  return v;
}

// The 8 entries of block b of a row of thresholds (q or keys), read into
// every lane by vector loads: they complete in order, so the next block's
// can be requested while this one is in use (scalar loads complete out of
// order, and waiting for one waits for all).
struct Q8 {
  uint4 lo, hi;
  __device__ uint32_t operator[](int j) const {
    const uint4& h = j < 4 ? lo : hi;
    const int i = j & 3;
    return i == 0 ? h.x : i == 1 ? h.y : i == 2 ? h.z : h.w;
  }
};
__device__ __forceinline__ Q8 load_q8(__amdgpu_buffer_rsrc_t rs, uint32_t row_bytes, int b) {
  // the offset is wave-uniform; stating it keeps it a scalar operand where
  // the compiler cannot prove it (else it loops over the lanes' values)
  const uint32_t off = __builtin_amdgcn_readfirstlane(row_bytes + 32u * (uint32_t)b);
  Q8 x;
  x.lo = load_mval<0>(rs, off);
  x.hi = load_mval<16>(rs, off);
  return x;
}

// Randomized rounding into mask row r of a group, lane = candidate. Word i
// of the row is the group's 64 decisions [u_{k,r,i} < q[r][i]] (the same
// draws as round_word); candidate 0 takes the deterministic bits under
// CKM_F_DET0. A block of 8 nodes shares one Philox output per lane.
// Philox4x32-10 of counter (b, r, k, 0), the counter of block b of row r for
// candidate k, split by what each part depends on. Round 0 multiplies b
// (wave-uniform) and k (per lane, the same for every block of the row);
// round 1 multiplies round 0's two results again. So the per-lane products
// of rounds 0 and 1 are made once per row (PhiloxRow), the per-block products
// are scalar, and a block costs each lane two XORs of round 1 and rounds 2-9.
struct PhiloxRow {
  uint32_t lo_k;          // lo(M1 k): round 0's counter word 1
  uint32_t hi_n, lo_n;    // M0 n0, n0 = hi(M1 k) ^ r ^ key0: round 1's product of word 0
};
__device__ __forceinline__ PhiloxRow philox_row(uint32_t r, uint32_t k, uint32_t key0) {
  const uint64_t a = (uint64_t)kPhiloxM1 * k;
  const uint32_t n0 = (uint32_t)(a >> 32) ^ (r ^ key0);
  const uint64_t p = (uint64_t)kPhiloxM0 * n0;
  return {(uint32_t)a, (uint32_t)(p >> 32), (uint32_t)p};
}
__device__ __forceinline__ void philox_block(const PhiloxRow& pr, uint32_t b, uint32_t key0, uint32_t key1,
                                             uint32_t x[4]) {
  // round 0: words 2, 3 from the block index alone
  const uint64_t pb = (uint64_t)kPhiloxM0 * b;
  const uint32_t w2 = (uint32_t)(pb >> 32) ^ key1, w3 = (uint32_t)pb;
  // round 1: word 2's product is uniform, word 0's was made per row
  uint32_t k0 = key0 + kPhiloxW0, k1 = key1 + kPhiloxW1;
  const uint64_t pu = (uint64_t)kPhiloxM1 * w2;
  uint32_t c0 = pr.lo_k ^ ((uint32_t)(pu >> 32) ^ k0);
  uint32_t c1 = (uint32_t)pu;
  uint32_t c2 = pr.hi_n ^ (w3 ^ k1);
  uint32_t c3 = pr.lo_n;
  // round 2: word 1 is still uniform
  k0 += kPhiloxW0;
  k1 += kPhiloxW1;
  {
    const uint64_t p0 = (uint64_t)kPhiloxM0 * c0;
    const uint64_t p1 = (uint64_t)kPhiloxM1 * c2;
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ (c1 ^ k0);
    const uint32_t n2 = xor3((uint32_t)(p0 >> 32), c3, k1);
    c0 = n0; c1 = (uint32_t)p1; c2 = n2; c3 = (uint32_t)p0;
  }
#pragma unroll
  for (int rr = 3; rr < 10; ++rr) {
    k0 += kPhiloxW0;
    k1 += kPhiloxW1;
    const uint64_t p0 = (uint64_t)kPhiloxM0 * c0;
    const uint64_t p1 = (uint64_t)kPhiloxM1 * c2;
    const uint32_t n0 = xor3((uint32_t)(p1 >> 32), c1, k0);
    const uint32_t n2 = xor3((uint32_t)(p0 >> 32), c3, k1);
    c0 = n0; c1 = (uint32_t)p1; c2 = n2; c3 = (uint32_t)p0;
  }
  x[0] = c0; x[1] = c1; x[2] = c2; x[3] = c3;
}

// Block b of row r (8 nodes) for the 64 candidates of a group, thresholds
// qb: one Philox output per lane, 8 compares whose lane masks are the words,
// one 64-byte store.
__device__ __forceinline__ void round_mask_block(const PhiloxRow& pr, const Q8& qb, int b, int r, uint32_t k,
                                                 uint32_t key0, uint32_t key1, bool det_here,
                                                 cptr<uint32_t> drow, uint32_t* dst) {
  uint64_t m[8];
  if (8 * b >= r) {
#pragma unroll
    for (int j = 0; j < 8; ++j) m[j] = 0ull;
  } else {
    uint32_t x[4];
    philox_block(pr, (uint32_t)b, key0, key1, x);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t u = (x[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
      m[j] = mask_of(u < qb[j]);
    }
    if (det_here) {
      const uint32_t dw = drow[b >> 2] >> (8 * (b & 3));
#pragma unroll
      for (int j = 0; j < 8; ++j) m[j] = (m[j] & ~1ull) | ((dw >> j) & 1u);
    }
  }
  // lanes 16-63 of out are never stored, so out starts from any value
  const uint32_t out = put_masks<0>(k, m);
  if (threadIdx.x < 16) dst[16 * b + threadIdx.x] = out;   // words 8b .. 8b+7 of the row
}

__device__ __forceinline__ void round_mask_row(const uint32_t* __restrict__ q, const uint32_t* __restrict__ det,
                                               int32_t n, int32_t ldq, int32_t det_words, uint32_t key0,
                                               uint32_t key1, uint32_t det0, int group, int r, uint64_t* row) {
  const int lane = threadIdx.x;
  const uint32_t k = (uint32_t)(group * kWave + lane);
  uint32_t* dst = reinterpret_cast<uint32_t*>(row);
  const int nblk = (r >> 3) + 1;
  const auto rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(q), 0, n * ldq * 4, kBufWord3);
  const uint32_t row_bytes = (uint32_t)(r < n ? r : 0) * (uint32_t)ldq * 4u;
  const cptr<uint32_t> drow = as_const(det + (size_t)(r < n ? r : 0) * det_words);
  const PhiloxRow pr = philox_row((uint32_t)r, k, key0);
  const bool det_here = det0 && group == 0;
  // two threshold buffers by block parity, each block's requested one block
  // ahead (vector loads complete in order)
  Q8 qa = load_q8(rs, row_bytes, 0), qb;
  for (int b = 0; b < nblk; b += 2) {
    if (b + 1 < nblk) qb = load_q8(rs, row_bytes, b + 1);
    round_mask_block(pr, qa, b, r, k, key0, key1, det_here, drow, dst);
    if (b + 1 >= nblk) break;
    if (b + 2 < nblk) qa = load_q8(rs, row_bytes, b + 2);
    round_mask_block(pr, qb, b + 1, r, k, key0, key1, det_here, drow, dst);
  }
}

// Block (group, y) makes row n - y of the group (rows 0 .. n; row n is
// zero). Blocks start in order of y, so the longest rows start first and the
// last to start are the shortest: the launch ends with little left on any
// SIMD. (Equal pairs of rows y and n - y per block ended with most SIMDs
// running one wave, the youngest, which the issue order serves last.)
__global__ void __launch_bounds__(kWave) ckm_round_masks_kernel(const uint32_t* __restrict__ q,
                                                                const uint32_t* __restrict__ det, int32_t n,
                                                                int32_t ldq, int32_t det_words, uint32_t key0,
                                                                uint32_t key1, uint32_t det0, size_t mgroup,
                                                                uint64_t* __restrict__ mrows, int32_t g0,
                                                                Totals tot) {
  const int group = blockIdx.x + g0;
  const int y = blockIdx.y;
  clear_totals(tot, group);
  uint64_t* rows = mrows + (size_t)group * mgroup;
  round_mask_row(q, det, n, ldq, det_words, key0, key1, det0, group, n - y, rows + mrow_off(n - y));
}

// ---------------------------------------------------------------------------
// Seen path: the mask path for graphs of up to 4096 nodes with any number of
// users and dependencies per node. What a node needs from users more than 32
// nodes above it goes through a per-lane "seen" bit of the used node: when a
// far user u of node x (u > x + 32) is decided, it ORs R_t[u] into x's seen
// bit. When the scan reaches x, the bit holds R_t of x's far users (all above
// it), and when a user v of x looks for users of x computed after v, the bit
// holds those of x's far users above v (a far user within 32 above v is also
// in v's R window). Near users stay in the window, as in the mask path. The
// seen bits are numbered over the nodes that have a far user, in order of
// their first far user: W words per lane in LDS (word w of lane j at byte
// 256 w + 4 j), cleared at each stage. Stage t writes only bits of nodes
// whose first far user is at most t, a prefix of that order, so the stages
// below a split point need only the first words: they run in a launch of
// their own with that much LDS (more waves per CU), where every read past
// those words lands on one more word that stays zero.
//
// Node v's data, 128 bytes at 128 v (v = 0 .. n; node n has only the fetch
// block for node n-1):
//   [0, 64)   record, 16 dwords (one scalar load):
//     0  users u of v with u <= v + 32 (bit u - v - 1)
//     1  v's seen bit (0 when v has no far user)
//     2  slots 2-3 present (bit 0) | overflow list present (bit 1) | its
//        length << 8
//     3  seen writes of slots 0 (low half) and 1 (high half): the LDS byte
//        offset of the dependency's seen word | kSWrite when v is a far user
//        of the dependency
//     4, 5  slot 0: lm (users u of the dependency with v < u <= v + 32, bit
//           u - v - 1), the dependency's seen bit (0: it has no far user)
//     6, 7  slot 1
//     8  first overflow entry (dependencies beyond the fourth)
//     fetch block, for node v-1 (all zero for v = 0):
//     9  byte offsets in a mask row of the S_{t+1} words of v-1's slot 0 and
//        1 dependencies (low, high half) | kSExtNext: v-1 has slots 2-3
//     10 the same for slots 2 and 3
//     11 128 (v - 1)
//     12 LDS byte offsets of v-1's seen word | of its slot 0 dependency's << 16
//     13 slot 1 | slot 2 << 16
//     14 slot 3
//     15 seen writes of slots 2 and 3 (as word 3)
//   [64, 112) binary64 M_v, C_v, M of slots 0-3
//   [112, 128) slots 2 and 3: lm, seen bit each
// An absent slot has lm = 0, no seen bit and size 0: it frees nothing.
// Overflow entries, 32 bytes: lm, seen bit, seen write (as word 3), byte
// offset of the S_{t+1} word, LDS byte offset of the seen word, M (binary64).
// All loads for node v-1 take their addresses from node v's record, so they
// are issued after it has arrived, one batch per node.
constexpr int kSNodeBytes = 128;
// Graphs with fewer seen words run every stage in one launch.
constexpr int32_t kSeenSplitMinWords = 16;
constexpr uint32_t kSExt = 1u, kSOver = 2u, kSWrite = 0x8000u, kSExtNext = 0x8000u;

struct SeenArgs {
  int32_t n, K, items, kind, P, T0, R1, R2;   // work plan (see Plan)
  int32_t np;                                 // node data entries: n + 1
  int32_t seen_words;                         // LDS words per lane of this launch
  uint32_t seen_lim;                          // byte offset of its last word: reads clamp to it
  int32_t item0;                              // work item of blockIdx.y = 0
  double base;                                // M_in + 2 M_param
  size_t mgroup;                              // words of one group's mask rows
  cptr<uint64_t> mrows;                       // S masks, group-major
  cptr<u32x16> snodes;                        // np x 128 bytes of node data
  cptr<u32x8> over;                           // overflow entries
  uint32_t* __restrict__ rrows;               // R rows out (row array layout)
  int32_t kpad;
  int64_t* __restrict__ part_peak;
  int64_t* __restrict__ part_cost;
  int32_t* __restrict__ hdr;
  int32_t g0;                                 // group of blockIdx.x = 0
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t snode_rsrc(const SeenArgs& a) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<u32x16*>((const u32x16*)a.snodes), 0, a.np * kSNodeBytes,
                                           kBufWord3);
}
// The lane's word at LDS byte offset off (off wave-uniform, a multiple of 256).
__device__ __forceinline__ uint32_t seen_read(const SeenArgs& a, char* lds_lane, uint32_t off) {
  return *reinterpret_cast<const uint32_t*>(lds_lane + min(off, a.seen_lim));
}
__device__ __forceinline__ void seen_or(char* lds_lane, uint32_t off, uint32_t bits) {
  atomicOr(reinterpret_cast<uint32_t*>(lds_lane + off), bits);
}

// What node v needs, all requested while node v+1 is decided.
struct SNode {
  u32x16 rec;
  uint64_t S0, S1;          // S_t[v], S_{t+1}[v]
  uint64_t d0, d1, d2, d3;  // S_{t+1} words of the slot 0-3 dependencies
  u32x4 ext;                // slots 2-3
  uint32_t has_ext;
  uint4 mc, dm, dm2;        // M_v, C_v | M of slots 0, 1 | M of slots 2, 3
  uint32_t sv, s0, s1, s2, s3;   // seen words of v and of the slot dependencies
};

__device__ __forceinline__ SNode seen_fetch(const SeenArgs& a, const u32x16& rec_v, cptr<uint64_t> s0row,
                                            cptr<uint64_t> s1row, char* lds_lane) {
  const uint32_t off = rec_v[11], f01 = rec_v[9];
  SNode nx;
  nx.rec = sload<u32x16>(a.snodes, off);
  nx.S0 = sload<uint64_t>(s0row, off >> 4);   // 8 (v - 1)
  nx.S1 = sload<uint64_t>(s1row, off >> 4);
  nx.d0 = sload<uint64_t>(s1row, f01 & 0x7FFFu);
  nx.d1 = sload<uint64_t>(s1row, f01 >> 16);
  const auto rs = snode_rsrc(a);
  nx.mc = load_mval<64>(rs, off);
  nx.dm = load_mval<80>(rs, off);
  nx.sv = seen_read(a, lds_lane, rec_v[12] & 0xFFFFu);
  nx.s0 = seen_read(a, lds_lane, rec_v[12] >> 16);
  nx.s1 = seen_read(a, lds_lane, rec_v[13] & 0xFFFFu);
  nx.has_ext = f01 & kSExtNext;
  if (nx.has_ext) {
    const uint32_t f23 = rec_v[10];
    nx.d2 = sload<uint64_t>(s1row, f23 & 0xFFFFu);
    nx.d3 = sload<uint64_t>(s1row, f23 >> 16);
    nx.ext = sload<u32x4>(a.snodes, off + 112);
    nx.dm2 = load_mval<96>(rs, off);
    nx.s2 = seen_read(a, lds_lane, rec_v[13] >> 16);
    nx.s3 = seen_read(a, lds_lane, rec_v[14]);
  }
  return nx;
}

struct SScan {
  double U0, Y, maxv, cost;
  uint32_t Rwin;   // R bits of nodes v+1 .. v+32 (bit d <-> node v + 1 + d)
};

// One dependency slot of node v (see mask_slot): later users of the
// dependency are those in v's R window (lm) and those its seen bit holds.
// Then, when v is a far user of the dependency, R_t[v] goes into its bit.
__device__ __forceinline__ double seen_slot(double val, uint64_t R, bool rb, uint32_t lm, uint32_t bit, uint32_t sw,
                                            uint64_t s1i, double Mi, uint32_t Rwin, uint32_t wr, char* lds_lane) {
  const uint32_t y = (Rwin & lm) | (sw & bit);
  const uint64_t later = mask_of(y != 0u);
  const uint64_t fr = R & ~(s1i | later);
  val = madd_m(val, fr, Mi);
  if (wr & kSWrite) seen_or(lds_lane, wr & 0x7FFFu, rb ? bit : 0u);
  return val;
}

// Node v of stage t (see mask_node and mask_node_as). kTop: v = t.
template <bool kTop, bool kSkip>
__device__ __forceinline__ void seen_node(const SeenArgs& a, const SNode& nd, cptr<uint64_t> s1row, SScan& sc,
                                          char* lds_lane) {
  const u32x16& r = nd.rec;
  const double Mv = dbl(nd.mc.x, nd.mc.y), Cv = dbl(nd.mc.z, nd.mc.w);
  const uint32_t x = (sc.Rwin & r[0]) | (nd.sv & r[1]);
  const uint64_t x1 = nd.S1 | mask_of(x != 0u);
  uint64_t R = x1 & ~nd.S0;
  sc.U0 = madd_m(sc.U0, nd.S0, Mv);
  if (kSkip && !kTop && R == 0ull) {
    sc.Rwin = sc.Rwin + sc.Rwin;   // no candidate computes v (see mask_node_as)
    return;
  }
  double val = sc.Y;
  if (kTop) {
    R = ~0ull;
    val = madd_m(val, ~x1, Mv);
  }
  const bool rb = lane_of(R);
  val = seen_slot(val, R, rb, r[4], r[5], nd.s0, nd.d0, dbl(nd.dm.x, nd.dm.y), sc.Rwin, r[3] & 0xFFFFu, lds_lane);
  val = seen_slot(val, R, rb, r[6], r[7], nd.s1, nd.d1, dbl(nd.dm.z, nd.dm.w), sc.Rwin, r[3] >> 16, lds_lane);
  if (nd.has_ext) {
    val = seen_slot(val, R, rb, nd.ext[0], nd.ext[1], nd.s2, nd.d2, dbl(nd.dm2.x, nd.dm2.y), sc.Rwin,
                    r[15] & 0xFFFFu, lds_lane);
    val = seen_slot(val, R, rb, nd.ext[2], nd.ext[3], nd.s3, nd.d3, dbl(nd.dm2.z, nd.dm2.w), sc.Rwin, r[15] >> 16,
                    lds_lane);
  }
  if (__builtin_expect((r[2] & kSOver) != 0u, 0)) {
    // dependencies beyond the fourth, one entry at a time
    const uint32_t cnt = r[2] >> 8;
    for (uint32_t c = 0, e = r[8]; c < cnt; ++c, ++e) {
      const u32x8 en = a.over[e];
      const uint64_t s1i = sload<uint64_t>(s1row, en[3]);
      const uint32_t sw = seen_read(a, lds_lane, en[4]);
      val = seen_slot(val, R, rb, en[0], en[1], sw, s1i, dbl(en[5], en[6]), sc.Rwin, en[2], lds_lane);
    }
  }
  // suffix form of the U recurrence (see scan_node): val = Y + freed_v
  sc.maxv = max_f64(sc.maxv, val);
  const double sel = rb ? 1.0 : 0.0;
  sc.Y = fma(-sel, Mv, val);
  sc.cost = fma(sel, Cv, sc.cost);
  sc.Rwin = sc.Rwin + sc.Rwin + (rb ? 1u : 0u);
}

// Node v from buf[P] (P: its parity in the scan), node v-1's loads into
// buf[P ^ 1] first.
template <int P, bool kTop, bool kSkip>
__device__ __forceinline__ void seen_step(const SeenArgs& a, int v, SNode (&buf)[2], cptr<uint64_t> s0row,
                                          cptr<uint64_t> s1row, SScan& sc, char* lds_lane, uint32_t* rrow_t) {
  buf[P ^ 1] = seen_fetch(a, buf[P].rec, s0row, s1row, lds_lane);
  seen_node<kTop, kSkip>(a, buf[P], s1row, sc, lds_lane);
  if ((v & 31) == 0) rrow_t[(size_t)(v >> 5) * a.kpad] = sc.Rwin;   // R of nodes v .. v+31
}

// One wave per work item: the 64 candidates of group blockIdx.x over the
// stages of item blockIdx.y; the scan of stage t runs from node t down.
template <bool kSkip>
__global__ void __launch_bounds__(kWave) ckm_seen_eval_kernel(SeenArgs a) {
  extern __shared__ uint32_t seen_lds[];
  const int lane = threadIdx.x;
  const int group = blockIdx.x + a.g0;
  const int item = blockIdx.y + a.item0;
  const uint32_t k = (uint32_t)(group * kWave + lane);
  char* lds_lane = reinterpret_cast<char*>(seen_lds) + 4 * lane;
  int t0, t1;
  item_range(a, item, t0, t1);
  const cptr<uint64_t> rows = a.mrows + (size_t)group * a.mgroup;
  double seg_peak = -INFINITY;
  int64_t seg_cost = 0;
  for (int t = t0; t < t1; ++t) {
    for (int w = 0; w < a.seen_words; ++w) *reinterpret_cast<uint32_t*>(lds_lane + 256 * w) = 0u;
    const cptr<uint64_t> s0row = rows + mrow_off(t);
    const cptr<uint64_t> s1row = rows + mrow_off(t + 1);
    uint32_t* rrow_t = a.rrows + row_base(t) * (size_t)a.kpad + k;
    SScan sc;
    sc.U0 = (double)a.base;
    sc.Y = 0.0;
    sc.maxv = -INFINITY;
    sc.cost = 0.0;
    sc.Rwin = 0u;
    SNode buf[2];
    const u32x16 top = a.snodes[(size_t)(t + 1) * (kSNodeBytes / 64)];   // its fetch block: node t
    buf[1] = seen_fetch(a, top, s0row, s1row, lds_lane);
    seen_step<1, true, kSkip>(a, t, buf, s0row, s1row, sc, lds_lane, rrow_t);
    int v = t - 1;
    for (; v >= 1; v -= 2) {
      seen_step<0, false, kSkip>(a, v, buf, s0row, s1row, sc, lds_lane, rrow_t);
      seen_step<1, false, kSkip>(a, v - 1, buf, s0row, s1row, sc, lds_lane, rrow_t);
    }
    if (v == 0) seen_step<0, false, kSkip>(a, 0, buf, s0row, s1row, sc, lds_lane, rrow_t);
    seg_peak = fmax(seg_peak, sc.U0 - sc.Y + sc.maxv);
    seg_cost += (int64_t)sc.cost;
  }
  if ((int)k < a.K && t0 < t1) {
    atomicMax(reinterpret_cast<long long*>(a.part_peak) + k, (long long)seg_peak);
    atomicAdd(reinterpret_cast<unsigned long long*>(a.part_cost) + k, (unsigned long long)seg_cost);
  }
  if (group == 0 && item == 0 && lane == 0) a.hdr[0] = a.items;
}

// Threshold candidates into mask rows (block (group, y): row n - y):
// word i of row r is the group's 64 decisions [rank_k < key[r][i]], the
// threshold test of threshold_word. Keys on and above the diagonal are 0, so
// are their words (row n reads row 0, all of whose keys are 0).
// Block b (8 nodes) of a threshold row: word i is the lane mask of
// [rank_k < key_i] (keys at and above the diagonal are 0).
__device__ __forceinline__ void threshold_mask_block(const Q8& kb, uint32_t rk, uint32_t k, int b, uint32_t* dst) {
  uint64_t m[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) m[j] = mask_of(rk < kb[j]);
  // lanes 16-63 of out are never stored, so out starts from any value
  const uint32_t out = put_masks<0>(k, m);
  if (threadIdx.x < 16) dst[16 * b + threadIdx.x] = out;
}

__global__ void __launch_bounds__(kWave) ckm_threshold_masks_kernel(const uint32_t* __restrict__ key, int32_t ldq,
                                                                    const uint32_t* __restrict__ rank, int32_t K,
                                                                    int32_t n, size_t mgroup,
                                                                    uint64_t* __restrict__ mrows, int32_t g0,
                                                                    Totals tot) {
  const int lane = threadIdx.x;
  const int group = blockIdx.x + g0;
  clear_totals(tot, group);
  const uint32_t k = (uint32_t)(group * kWave + lane);
  const uint32_t rk = rank[k < (uint32_t)K ? k : (uint32_t)K - 1u];
  uint64_t* rows = mrows + (size_t)group * mgroup;
  const auto rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(key), 0, n * ldq * 4, kBufWord3);
  // row n - y (longest first, as in ckm_round_masks_kernel); the row is
  // wave-uniform, and stating it keeps the block loop scalar
  const int r = __builtin_amdgcn_readfirstlane(n - (int)blockIdx.y);
  uint32_t* dst = reinterpret_cast<uint32_t*>(rows + mrow_off(r));
  const int lim = r < n ? r : 0;   // row n (after the last stage) is empty
  const uint32_t rb = (uint32_t)lim * (uint32_t)ldq * 4u;
  const int nblk = (r >> 3) + 1;
  // two key buffers by block parity, each block's requested one block ahead
  Q8 ka = load_q8(rs, rb, 0), kb;
  for (int b = 0; b < nblk; b += 2) {
    if (b + 1 < nblk) kb = load_q8(rs, rb, b + 1);
    threshold_mask_block(ka, rk, k, b, dst);
    if (b + 1 >= nblk) break;
    if (b + 2 < nblk) ka = load_q8(rs, rb, b + 2);
    threshold_mask_block(kb, rk, k, b + 1, dst);
  }
}

// Caller-supplied checkpoint matrices into mask rows (block (group, y): row
// n - y): word i of row r is bit i of row r of each of the group's 64
// matrices ([K][n][s_words] 32-bit words), for i < r only (bits on and above
// the diagonal are not part of S). Lanes past K repeat candidate K-1. Each
// lane reads its matrix row 16 bytes (128 nodes) at a time, the next chunk
// requested before the current one is turned into masks.
__device__ __forceinline__ uint4 user_chunk(const uint32_t* row, int c, int lim) {
  // chunk c: words 4c .. 4c+3; only words with a node below lim are read
  uint4 x = make_uint4(0u, 0u, 0u, 0u);
  if (128 * c < lim) x.x = row[4 * c];
  if (128 * c + 32 < lim) x.y = row[4 * c + 1];
  if (128 * c + 64 < lim) x.z = row[4 * c + 2];
  if (128 * c + 96 < lim) x.w = row[4 * c + 3];
  return x;
}

__global__ void __launch_bounds__(kWave) ckm_user_masks_kernel(const uint32_t* __restrict__ s_user, int32_t n,
                                                               int32_t K, int32_t s_words, size_t mgroup,
                                                               uint64_t* __restrict__ mrows, int32_t g0,
                                                               Totals tot) {
  const int lane = threadIdx.x;
  const int group = blockIdx.x + g0;
  clear_totals(tot, group);
  const uint32_t k = (uint32_t)(group * kWave + lane);
  const uint32_t kk = k < (uint32_t)K ? k : (uint32_t)K - 1u;
  uint64_t* rows = mrows + (size_t)group * mgroup;
  // row n - y (longest first, as in ckm_round_masks_kernel); the row is
  // wave-uniform, and stating it keeps the block loop scalar
  const int r = __builtin_amdgcn_readfirstlane(n - (int)blockIdx.y);
  uint32_t* dst = reinterpret_cast<uint32_t*>(rows + mrow_off(r));
  const int lim = r < n ? r : 0;   // row n (after the last stage) is empty
  const uint32_t* src = s_user + ((size_t)kk * n + lim) * s_words;
  const int nblk = (r >> 3) + 1;
  uint4 cur = user_chunk(src, 0, lim);
  for (int c = 0; 16 * c < nblk; ++c) {
    const uint4 nxt = user_chunk(src, c + 1, lim);
    const uint32_t w4[4] = {cur.x, cur.y, cur.z, cur.w};
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int b = 16 * c + q;
      if (b >= nblk) break;
      // the block's bits of nodes below lim only
      const int below = lim - 8 * b;
      const uint32_t keep = below >= 8 ? 0xFFu : below <= 0 ? 0u : (1u << below) - 1u;
      const uint32_t byte = (w4[q >> 2] >> (8 * (q & 3))) & keep;
      uint64_t m[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) m[j] = mask_of(((byte >> j) & 1u) != 0u);
      const uint32_t out = put_masks<0>(k, m);   // lanes 16-63 are not stored
      if (lane < 16) dst[16 * b + lane] = out;
    }
    cur = nxt;
  }
}

template <typename T>
T* at(char* work, size_t off) { return reinterpret_cast<T*>(work + off); }

}  // namespace

// ---------------------------------------------------------------------------
hipError_t launch_quantize(const ckm_graph& g, const Layout& L, const double* d_s, int64_t ld,
                           char* work, hipStream_t stream) {
  hipLaunchKernelGGL(ckm_quantize_kernel, dim3(g.n), dim3(256), 0, stream, d_s, ld, g.n, L.ldq,
                     L.det_words, at<uint32_t>(work, L.q_off), at<uint32_t>(work, L.det_off),
                     at<int32_t>(work, L.nan_off));
  return hipGetLastError();
}

hipError_t launch_threshold_keys(const ckm_graph& g, const Layout& L, const double* d_s, int64_t ld,
                                 const double* d_p, int32_t K, char* work, hipStream_t stream) {
  double* sorted = at<double>(work, L.thr_sorted_off);
  hipLaunchKernelGGL(ckm_threshold_rank_kernel, dim3((K + 255) / 256), dim3(256), 0, stream, K, d_p, sorted,
                     at<uint32_t>(work, L.thr_rank_off));
  hipLaunchKernelGGL(ckm_threshold_key_kernel, dim3(g.n), dim3(256), 0, stream, d_s, ld, g.n, L.ldq, K, d_p,
                     static_cast<const double*>(sorted), at<uint32_t>(work, L.q_off),
                     at<int32_t>(work, L.nan_off));
  return hipGetLastError();
}

// Width of the register row for rows of `words` 32-bit words (0: LDS rows).
static int reg_row_width(int32_t words) {
  return words <= 32 ? 32 : words <= 64 ? 64 : words <= 128 ? 128 : 0;
}

template <int kSrc>
static void (*eval_kernel_w(int w))(EvalArgs) {
  switch (w) {
    case 32: return ckm_eval_kernel<32, kSrc>;
    case 64: return ckm_eval_kernel<64, kSrc>;
    case 128: return ckm_eval_kernel<128, kSrc>;
    default: return ckm_eval_kernel<0, kSrc>;
  }
}

// Wide graphs (int64 sums) use the LDS-row variant only: they are rare, and
// one variant per row source keeps the library small.
static void (*eval_kernel_for(int32_t words, int src, bool wide))(EvalArgs) {
  if (wide) {
    if (src == kSrcRows) return ckm_eval_kernel<0, kSrcRows, true>;
    if (src == kSrcUser) return ckm_eval_kernel<0, kSrcUser, true>;
    if (src == kSrcThreshold) return ckm_eval_kernel<0, kSrcThreshold, true>;
    return ckm_eval_kernel<0, kSrcRound, true>;
  }
  const int w = reg_row_width(words);
  if (src == kSrcRows) return eval_kernel_w<kSrcRows>(w);
  if (src == kSrcUser) return eval_kernel_w<kSrcUser>(w);
  if (src == kSrcThreshold) return eval_kernel_w<kSrcThreshold>(w);
  return eval_kernel_w<kSrcRound>(w);
}

static size_t eval_lds_bytes(int32_t words, bool wide) {
  return (!wide && reg_row_width(words) ? 1u : 2u) * (size_t)words * kWave * sizeof(uint32_t);
}

int32_t eval_waves_per_cu(int32_t n, bool wide) {
  const int32_t words = (n >> 5) + 1;
  const void* fn = (const void*)eval_kernel_for(words, kSrcRound, wide);
  const size_t lds = eval_lds_bytes(words, wide);
  if (lds > 65536) (void)hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, fn, kWave, lds) != hipSuccess || blocks < 1) blocks = 1;
  return blocks;
}

static unsigned groups_of(int32_t K) { return (unsigned)((K + kWave - 1) / kWave); }

static bool use_mask_path(const ckm_graph& g, const Layout& L) {
  return L.rows_on && (g.d_mrecs != nullptr || g.d_snodes != nullptr);
}

int32_t mask_waves_per_cu() {
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, (const void*)ckm_mask_eval_kernel<false>, kWave, 0) !=
          hipSuccess ||
      blocks < 1)
    blocks = 1;
  return blocks;
}

int32_t seen_waves_per_cu(int32_t seen_words) {
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, (const void*)ckm_seen_eval_kernel<false>, kWave,
                                                   (size_t)seen_words * 256) != hipSuccess ||
      blocks < 1)
    blocks = 1;
  return blocks;
}

size_t mask_rows_words(int32_t n) { return mrow_off(n + 1); }

hipError_t launch_round_rows(const ckm_graph& g, const Layout& L, int32_t K, uint64_t seed, uint32_t flags,
                             char* work, hipStream_t stream) {
  return launch_round_rows(g, L, K, seed, flags, 0, (int32_t)groups_of(K), false, work, stream);
}

hipError_t launch_round_rows(const ckm_graph& g, const Layout& L, int32_t K, uint64_t seed, uint32_t flags,
                             int32_t g0, int32_t gn, bool clear, char* work, hipStream_t stream) {
  if (!L.rows_on || gn <= 0) return hipSuccess;
  if (use_mask_path(g, L)) {
    const Totals tot{clear ? at<int64_t>(work, L.part_peak_off) : nullptr, at<int64_t>(work, L.part_cost_off), K};
    hipLaunchKernelGGL(ckm_round_masks_kernel, dim3(gn, g.n + 1), dim3(kWave), 0, stream,
                       at<const uint32_t>(work, L.q_off), at<const uint32_t>(work, L.det_off), g.n, L.ldq,
                       L.det_words, (uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32),
                       (flags & CKM_F_DET0) ? 1u : 0u, mask_rows_words(g.n), at<uint64_t>(work, L.rows_off), g0,
                       tot);
    return hipGetLastError();
  }
  const int32_t kpad = ((K + kWave - 1) / kWave) * kWave;
  hipLaunchKernelGGL(ckm_round_rows_kernel, dim3((K + kWave - 1) / kWave, g.n), dim3(kWave), 0, stream,
                     at<const uint32_t>(work, L.q_off), at<const uint32_t>(work, L.det_off), L.ldq, L.det_words,
                     (uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32), (flags & CKM_F_DET0) ? 1u : 0u, kpad,
                     at<uint32_t>(work, L.rows_off));
  return hipGetLastError();
}

// Overlapped launches (seen path, when LDS holds its evaluate to at most
// kForkMaxWaves waves per CU). The first quarter of the candidate groups has
// its mask rows made alone; the other groups' producer then runs beside the
// first quarter's evaluate, and their evaluate follows on the side stream.
// The producers are VALU-bound, and an evaluate that LDS keeps at a few waves
// per SIMD leaves them registers and VALU slots: at n = 4001, K = 4096 (16 KiB
// of seen bits per wave, 10 waves per CU) the step drops from 95.3 to
// 91.7 ms (halves: 93.7, eighths: 91.3). An evaluate that its registers
// keep at 6 waves per SIMD leaves no room, and the second chunk's longest
// stages then start behind its producer: n = 1009, K = 1024 on the mask
// kernel takes 0.68 to 0.73 ms split against 0.611, n = 337, K = 512 on the
// seen kernel 0.156 against 0.106.
static int32_t fork_first_groups(int32_t groups) { return groups / 4 > 0 ? groups / 4 : 1; }
constexpr int32_t kForkMinGroups = 8;

hipError_t fork_create(Fork& f) {
  hipError_t e = hipStreamCreateWithFlags(&f.side, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&f.forked, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&f.joined, hipEventDisableTiming);
  if (e != hipSuccess) fork_destroy(f);
  return e;
}

void fork_destroy(Fork& f) {
  if (f.side) (void)hipStreamSynchronize(f.side);   // nothing of the graph's still running there
  if (f.forked) (void)hipEventDestroy(f.forked);
  if (f.joined) (void)hipEventDestroy(f.joined);
  if (f.side) (void)hipStreamDestroy(f.side);
  f.forked = f.joined = nullptr;
  f.side = nullptr;
}

// The mask rows of groups g0 .. g0 + gn - 1 from source src (kSrcRound,
// kSrcThreshold or kSrcUser); their candidates' totals are cleared on the
// way (the evaluate that follows accumulates into them).
static hipError_t launch_mask_producer(const ckm_graph& g, const Layout& L, int32_t K, uint64_t seed,
                                       uint32_t flags, int src, const uint64_t* s_user, int32_t g0, int32_t gn,
                                       char* work, hipStream_t stream) {
  if (gn <= 0) return hipSuccess;
  const Totals tot{at<int64_t>(work, L.part_peak_off), at<int64_t>(work, L.part_cost_off), K};
  if (src == kSrcThreshold) {
    hipLaunchKernelGGL(ckm_threshold_masks_kernel, dim3(gn, g.n + 1), dim3(kWave), 0, stream,
                       at<const uint32_t>(work, L.q_off), L.ldq, at<const uint32_t>(work, L.thr_rank_off), K, g.n,
                       mask_rows_words(g.n), at<uint64_t>(work, L.rows_off), g0, tot);
  } else if (src == kSrcUser) {
    hipLaunchKernelGGL(ckm_user_masks_kernel, dim3(gn, g.n + 1), dim3(kWave), 0, stream,
                       reinterpret_cast<const uint32_t*>(s_user), g.n, K, L.row_words, mask_rows_words(g.n),
                       at<uint64_t>(work, L.rows_off), g0, tot);
  } else {
    return launch_round_rows(g, L, K, seed, flags, g0, gn, true, work, stream);
  }
  return hipGetLastError();
}

// The mask-path evaluate (seen kernel or mask kernel) of groups g0 .. g0 + gn - 1.
// The evaluate of groups g0 .. g0 + gn - 1 on the mask rows. Rows of the
// threshold family or of supplied schedules take the kernels that skip a
// node no candidate of the group computes (see mask_node_as).
static hipError_t launch_mask_eval(const ckm_graph& g, const Layout& L, int32_t K, const Plan& plan, int src,
                                   int32_t g0, int32_t gn, char* work, hipStream_t stream) {
  if (gn <= 0) return hipSuccess;
  const bool skip = src != kSrcRound;
  const int32_t kpad = ((K + kWave - 1) / kWave) * kWave;
  if (g.d_snodes) {
    SeenArgs m;
    m.n = g.n;
    m.K = K;
    m.items = plan.items;
    m.kind = plan.kind;
    m.P = plan.P;
    m.T0 = plan.T0;
    m.R1 = plan.R1;
    m.R2 = plan.R2;
    m.np = g.n + 1;
    m.base = (double)g.base;
    m.mgroup = mask_rows_words(g.n);
    m.mrows = as_const(at<const uint64_t>(work, L.rows_off));
    m.snodes = (cptr<u32x16>)(g.d_snodes);
    m.over = (cptr<u32x8>)(g.d_sover);
    m.rrows = at<uint32_t>(work, L.rrows_off);
    m.kpad = kpad;
    m.part_peak = at<int64_t>(work, L.part_peak_off);
    m.part_cost = at<int64_t>(work, L.part_cost_off);
    m.hdr = at<int32_t>(work, L.hdr_off);
    m.g0 = g0;
    // items [i0, i0 + ni) with `words` LDS words per lane, reads clamped to
    // the last of them
    auto launch = [&](int32_t i0, int32_t ni, int32_t words) {
      m.item0 = i0;
      m.seen_words = words;
      m.seen_lim = (uint32_t)(words - 1) * 256u;
      if (skip)
        hipLaunchKernelGGL(ckm_seen_eval_kernel<true>, dim3(gn, ni), dim3(kWave), (size_t)words * 256, stream, m);
      else
        hipLaunchKernelGGL(ckm_seen_eval_kernel<false>, dim3(gn, ni), dim3(kWave), (size_t)words * 256, stream, m);
      return hipGetLastError();
    };
    // Items are numbered from stage n-1 down, one stage each above T0: the
    // stages at or above the first tier's split point take every word; those
    // below a tier's split point only that tier's words, plus one that stays
    // zero. A split point among the multi-stage items below T0 ends the tiers.
    if (g.seen_tiers > 0 && plan.kind == 1 && plan.P == 1) {
      int32_t i0 = 0, words = g.seen_words;
      hipError_t e = hipSuccess;
      for (int i = 0; i < g.seen_tiers && e == hipSuccess; ++i) {
        const int32_t ts = g.seen_tier_t[i];
        if (ts < plan.T0 || ts >= g.n) break;
        const int32_t iend = g.n - ts;
        if (iend > i0) {
          e = launch(i0, iend - i0, words);
          i0 = iend;
        }
        words = g.seen_tier_w[i] + 1;
      }
      if (e == hipSuccess && i0 < plan.items) e = launch(i0, plan.items - i0, words);
      return e;
    }
    return launch(0, plan.items, g.seen_words);
  }
  MaskArgs m;
  m.n = g.n;
  m.K = K;
  m.items = plan.items;
  m.kind = plan.kind;
  m.P = plan.P;
  m.T0 = plan.T0;
  m.R1 = plan.R1;
  m.R2 = plan.R2;
  m.base = (double)g.base;
  m.mgroup = mask_rows_words(g.n);
  m.mrows = as_const(at<const uint64_t>(work, L.rows_off));
  m.np = mask_padded_nodes(g.n);
  m.mnodes = (cptr<u32x16>)(g.d_mrecs);
  m.rrows = at<uint32_t>(work, L.rrows_off);
  m.kpad = kpad;
  m.part_peak = at<int64_t>(work, L.part_peak_off);
  m.part_cost = at<int64_t>(work, L.part_cost_off);
  m.hdr = at<int32_t>(work, L.hdr_off);
  m.g0 = g0;
  if (skip)
    hipLaunchKernelGGL(ckm_mask_eval_kernel<true>, dim3(gn, plan.items), dim3(kWave), 0, stream, m);
  else
    hipLaunchKernelGGL(ckm_mask_eval_kernel<false>, dim3(gn, plan.items), dim3(kWave), 0, stream, m);
  return hipGetLastError();
}

hipError_t launch_evaluate(const ckm_graph& g, const Layout& L, int32_t K, uint64_t seed,
                           uint32_t flags, const Plan& plan, int src, const uint64_t* s_user, char* work,
                           hipStream_t stream, bool overlap) {
  if (use_mask_path(g, L)) {
    // mask rows made by a producer (none when the caller rounded them
    // beforehand), then the evaluate, chunk by chunk
    const bool produce = !(src == kSrcRound && (flags & CKM_F_ROUNDED));
    const int32_t G = (int32_t)groups_of(K);
    hipError_t e = hipSuccess;
    if (!produce) {
      // no producer to clear the totals on the way
      hipLaunchKernelGGL(ckm_eval_init_kernel, dim3((K + 255) / 256), dim3(256), 0, stream, K,
                         at<int64_t>(work, L.part_peak_off), at<int64_t>(work, L.part_cost_off));
      e = hipGetLastError();
      if (e != hipSuccess) return e;
    }
    if (!(overlap && produce && g.fork && g.d_snodes && g.eval_waves <= kForkMaxWaves && G >= kForkMinGroups)) {
      if (produce) e = launch_mask_producer(g, L, K, seed, flags, src, s_user, 0, G, work, stream);
      if (e == hipSuccess) e = launch_mask_eval(g, L, K, plan, src, 0, G, work, stream);
      return e;
    }
    const int32_t ga = fork_first_groups(G);
    e = launch_mask_producer(g, L, K, seed, flags, src, s_user, 0, ga, work, stream);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lk(g.fork->mu);
    e = hipEventRecord(g.fork->forked, stream);
    if (e == hipSuccess) e = hipStreamWaitEvent(g.fork->side, g.fork->forked, 0);
    if (e == hipSuccess) e = launch_mask_producer(g, L, K, seed, flags, src, s_user, ga, G - ga, work, g.fork->side);
    if (e == hipSuccess) e = launch_mask_eval(g, L, K, plan, src, ga, G - ga, work, g.fork->side);
    if (e == hipSuccess) e = hipEventRecord(g.fork->joined, g.fork->side);
    // the first chunk's evaluate is enqueued whatever happened above, and the
    // caller's stream always waits for what the side stream was given
    hipError_t e2 = launch_mask_eval(g, L, K, plan, src, 0, ga, work, stream);
    hipError_t e3 = hipStreamWaitEvent(stream, g.fork->joined, 0);
    return e != hipSuccess ? e : e2 != hipSuccess ? e2 : e3;
  }
  EvalArgs a;
  a.n = g.n;
  a.K = K;
  a.s_user = reinterpret_cast<const uint32_t*>(s_user);
  a.s_words = L.row_words;
  a.rank = at<const uint32_t>(work, L.thr_rank_off);
  a.rows = at<const uint32_t>(work, L.rows_off);
  a.rrows = L.rows_on ? at<uint32_t>(work, L.rrows_off) : nullptr;
  a.kpad = ((K + kWave - 1) / kWave) * kWave;
  if (src == kSrcRound && L.rows_on) {
    // every row rounded once (here, or by an earlier launch_round_rows), then streamed
    if (!(flags & CKM_F_ROUNDED)) {
      hipError_t e = launch_round_rows(g, L, K, seed, flags, work, stream);
      if (e != hipSuccess) return e;
    }
    src = kSrcRows;
  } else if (src == kSrcThreshold && L.rows_on) {
    // threshold rows made once, then streamed
    hipLaunchKernelGGL(ckm_threshold_rows_kernel, dim3(groups_of(K), g.n), dim3(kWave), 0, stream,
                       at<const uint32_t>(work, L.q_off), L.ldq, at<const uint32_t>(work, L.thr_rank_off), K,
                       a.kpad, at<uint32_t>(work, L.rows_off));
    src = kSrcRows;
  } else if (src == kSrcUser && L.rows_on) {
    // the caller's rows transposed once into the streamed layout (reading
    // them in place puts each lane of a load in another candidate's matrix)
    const size_t tile = (size_t)(((g.n - 1) >> 5) + 1) * (kWave + 1) * sizeof(uint32_t);
    hipLaunchKernelGGL(ckm_user_rows_kernel, dim3(groups_of(K), g.n), dim3(256), tile, stream, a.s_user, g.n, K,
                       a.s_words, a.kpad, at<uint32_t>(work, L.rows_off));
    src = kSrcRows;
  }
  a.items = plan.items;
  a.kind = plan.kind;
  a.P = plan.P;
  a.T0 = plan.T0;
  a.R1 = plan.R1;
  a.R2 = plan.R2;
  a.ldq = L.ldq;
  a.det_words = L.det_words;
  a.row_words = (g.n >> 5) + 1;   // words for nodes 0 .. n (node n's bit is the "none" bit)
  a.key0 = (uint32_t)(seed & 0xFFFFFFFFu);
  a.key1 = (uint32_t)(seed >> 32);
  a.det0 = (flags & CKM_F_DET0) ? 1u : 0u;
  a.base = g.base;
  a.q = as_const(at<const uint32_t>(work, L.q_off));
  a.det = as_const(at<const uint32_t>(work, L.det_off));
  a.M = as_const(g.d_M);
  a.user_ptr = as_const(g.d_user_ptr);
  a.user_idx = as_const(g.d_user_idx);
  a.dep_ptr = as_const(g.d_dep_ptr);
  a.dep_idx = as_const(g.d_dep_idx);
  a.dep_upos = as_const(g.d_dep_upos);
  a.recs = reinterpret_cast<const uint4*>(g.d_recs);
  a.part_peak = at<int64_t>(work, L.part_peak_off);
  a.part_cost = at<int64_t>(work, L.part_cost_off);
  a.hdr = at<int32_t>(work, L.hdr_off);
  const int groups = (K + kWave - 1) / kWave;
  void (*fn)(EvalArgs) = eval_kernel_for(a.row_words, src, g.wide);
  const size_t lds_bytes = eval_lds_bytes(a.row_words, g.wide);
  if (lds_bytes > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(ckm_eval_init_kernel, dim3((K + 255) / 256), dim3(256), 0, stream, K, a.part_peak,
                     a.part_cost);
  hipLaunchKernelGGL(fn, dim3(groups, plan.items), dim3(kWave), lds_bytes, stream, a);
  return hipGetLastError();
}

static hipError_t launch_closure(const ckm_graph& g, const Layout& L, const int32_t* d_best_k,
                                 const uint32_t* S_base, size_t cand_stride, uint32_t* R_rows, hipStream_t stream) {
  ClosureArgs c;
  c.n = g.n;
  c.row_words = L.row_words;
  c.user_ptr = g.d_user_ptr;
  c.user_idx = g.d_user_idx;
  c.recs = reinterpret_cast<const uint4*>(g.d_recs);
  c.best_k = d_best_k;
  c.S_base = S_base;
  c.cand_stride = cand_stride;
  c.R_rows = R_rows;
  const size_t lds = (size_t)3 * ((g.n >> 5) + 1) * kWave * sizeof(uint32_t);
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute((const void*)ckm_best_closure_kernel,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(ckm_best_closure_kernel, dim3((g.n + kWave - 1) / kWave), dim3(kWave), lds, stream, c);
  return hipGetLastError();
}

hipError_t launch_max_batch(const ckm_graph& g, const Layout& L, int32_t K, int64_t budget, int64_t cost_cap,
                            int64_t* d_batch, int32_t* d_best_k, int64_t* d_best_batch, int32_t* d_status,
                            char* work, hipStream_t stream) {
  const int rb = L.reduce_blocks;
  hipLaunchKernelGGL(ckm_batch_kernel, dim3(rb), dim3(256), 0, stream, K, at<const int64_t>(work, L.part_peak_off),
                     at<const int64_t>(work, L.part_cost_off), g.base, budget, cost_cap, d_batch,
                     at<BestB>(work, L.bbest_off));
  hipLaunchKernelGGL(ckm_batch_argmax_kernel, dim3(1), dim3(256), 0, stream, rb, at<const BestB>(work, L.bbest_off),
                     g.n, at<const int32_t>(work, L.nan_off), d_best_k, d_best_batch, d_status);
  return hipGetLastError();
}

hipError_t launch_select(const ckm_graph& g, const Layout& L, int32_t K, uint64_t seed,
                         int64_t budget, uint32_t flags, int64_t* d_peak, int64_t* d_cost,
                         uint8_t* d_feasible, int32_t* d_best_k, uint64_t* d_best_S,
                         uint64_t* d_best_R, int32_t* d_status, int src, const uint64_t* s_user,
                         char* work, hipStream_t stream) {
  // rounded candidates: NaN flags from the quantize or key stage; supplied S: none
  const int32_t nan_rows = src == kSrcUser ? 0 : g.n;
  if (K <= kSelectOneBlock) {
    hipLaunchKernelGGL(ckm_select_kernel, dim3(1), dim3(1024), 0, stream, K,
                       at<const int64_t>(work, L.part_peak_off), at<const int64_t>(work, L.part_cost_off), budget,
                       d_peak, d_cost, d_feasible, nan_rows, at<const int32_t>(work, L.nan_off), d_best_k, d_status);
  } else {
    const int rb = L.reduce_blocks;
    hipLaunchKernelGGL(ckm_reduce_kernel, dim3(rb), dim3(256), 0, stream, K,
                       at<const int64_t>(work, L.part_peak_off), at<const int64_t>(work, L.part_cost_off),
                       budget, d_peak, d_cost, d_feasible, at<Best>(work, L.best_off));
    hipLaunchKernelGGL(ckm_argmin_kernel, dim3(1), dim3(256), 0, stream, rb,
                       at<const Best>(work, L.best_off), nan_rows, at<const int32_t>(work, L.nan_off), d_best_k,
                       d_status);
  }
  // With the row arrays the evaluate stage kept every candidate's R rows, so
  // the best R is a gather; otherwise Algorithm 2 runs again for it.
  const bool gather_R = d_best_R && L.rows_on;
  const int32_t kpad = (int32_t)(groups_of(K) * kWave);
  const dim3 rows_grid((L.row_words + 255) / 256, g.n);
  uint32_t* R_out = reinterpret_cast<uint32_t*>(d_best_R);
  if (src == kSrcUser) {
    if (gather_R) {
      hipLaunchKernelGGL(ckm_best_rrows_kernel, rows_grid, dim3(256), 0, stream,
                         at<const uint32_t>(work, L.rrows_off), kpad, L.row_words, d_best_k, R_out);
    } else if (d_best_R) {
      hipError_t e = launch_closure(g, L, d_best_k, reinterpret_cast<const uint32_t*>(s_user),
                                    (size_t)g.n * L.row_words, R_out, stream);
      if (e != hipSuccess) return e;
    }
  } else if (d_best_S || d_best_R) {
    // the S rows: output, and the closure's input when there is no gather
    uint32_t* srows = d_best_S ? reinterpret_cast<uint32_t*>(d_best_S) : at<uint32_t>(work, L.srows_off);
    hipLaunchKernelGGL(ckm_best_rows_kernel, rows_grid, dim3(256), 0, stream,
                       at<const uint32_t>(work, L.q_off), at<const uint32_t>(work, L.det_off), g.n,
                       L.ldq, L.det_words, L.row_words, (uint32_t)(seed & 0xFFFFFFFFu),
                       (uint32_t)(seed >> 32), (flags & CKM_F_DET0) ? 1u : 0u,
                       src == kSrcThreshold ? at<const uint32_t>(work, L.thr_rank_off) : nullptr, d_best_k,
                       srows, at<const uint32_t>(work, L.rrows_off), kpad, gather_R ? R_out : nullptr);
    if (d_best_R && !gather_R) {
      hipError_t e = launch_closure(g, L, d_best_k, static_cast<const uint32_t*>(srows), (size_t)0, R_out, stream);
      if (e != hipSuccess) return e;
    }
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// The second form of slow node v's lists (see kDwExt) into the record's
// dwords, or false when v exceeds its counts.
// A size or cost in the record's form: binary64, or int64 for a wide graph.
static uint64_t rec_value(int64_t x, bool wide) {
  if (wide) return (uint64_t)x;
  const double d = (double)x;
  uint64_t bits;
  memcpy(&bits, &d, sizeof(bits));
  return bits;
}

static bool build_ext_lists(int32_t v, const int64_t* M, bool wide, const int32_t* dep_ptr, const int32_t* dep_idx,
                            const int32_t* user_ptr, const int32_t* user_idx, uint32_t dw[64]) {
  auto put16 = [&](int at, int f, uint32_t node) { dw[at + f / 2] |= node << (16 * (f & 1)); };
  int nfar = 0;
  for (int32_t e = user_ptr[v]; e < user_ptr[v + 1]; ++e) {
    const int u = user_idx[e];
    if (u - v - 1 < 32) continue;
    if (nfar == kExtFar) return false;
    put16(kDwExt + 1, nfar++, (uint32_t)u);
  }
  const int nd = dep_ptr[v + 1] - dep_ptr[v];
  if (nd > kExtDeps) return false;
  for (int d = 0; d < nd; ++d) {
    const int i = dep_idx[dep_ptr[v] + d];
    const int b = ext_slot(d);
    uint32_t lm = 0;
    int nl = 0;
    for (int32_t e = user_ptr[i]; e < user_ptr[i + 1]; ++e) {
      const int u = user_idx[e];
      if (u <= v) continue;
      if (u - v - 1 < 32) {
        lm |= 1u << (u - v - 1);
      } else {
        if (nl == kExtLate) return false;
        put16(b + 4, nl++, (uint32_t)u);
      }
    }
    const uint64_t mbits = rec_value(M[i], wide);
    dw[b] = lm;
    dw[b + 1] = (uint32_t)mbits;
    dw[b + 2] = (uint32_t)(mbits >> 32);
    dw[b + 3] = (uint32_t)i | (uint32_t)nl << 16;
  }
  dw[kDwExt] = (uint32_t)nfar | (uint32_t)nd << 8 | kExtValid;
  return true;
}

int32_t mask_records_bytes(int32_t n) { return mask_padded_nodes(n) * kMNodeBytes; }

bool build_mask_records(int32_t n, const int64_t* M, const int64_t* C, const int32_t* dep_ptr,
                        const int32_t* dep_idx, const int32_t* user_ptr, const int32_t* user_idx, void* out) {
  const int32_t np = mask_padded_nodes(n);
  char* base = static_cast<char*>(out);
  memset(out, 0, (size_t)mask_records_bytes(n));
  auto far = [](int u) { return (uint32_t)u << 16 | (uint32_t)(u & 31); };
  auto put = [](uint32_t* w, double x) { memcpy(w, &x, sizeof(x)); };
  for (int32_t v = 0; v < np; ++v) {   // no far references, padded nodes included
    uint32_t* r = reinterpret_cast<uint32_t*>(base + (size_t)v * kMNodeBytes);
    r[1] = r[3] = r[5] = r[7] = r[16 + 1] = r[16 + 3] = kMNoFar;
  }
  for (int32_t v = 0; v < n; ++v) {
    char* node = base + (size_t)v * kMNodeBytes;
    uint32_t* r = reinterpret_cast<uint32_t*>(node);
    uint32_t* r2 = reinterpret_cast<uint32_t*>(node + 64);
    uint32_t* m23 = reinterpret_cast<uint32_t*>(node + 96);
    uint32_t ctrl = kMNoFar;   // stays, or names the one far user
    int nfar = 0;
    for (int32_t e = user_ptr[v]; e < user_ptr[v + 1]; ++e) {
      const int u = user_idx[e];
      if (u - v - 1 < 32) {
        r[0] |= 1u << (u - v - 1);
      } else {
        if (nfar++) return false;
        ctrl = far(u);
      }
    }
    const int nd = dep_ptr[v + 1] - dep_ptr[v];
    if (nd > 4) return false;
    if (nd > 2) {
      ctrl |= kMRare;
      r2[4] = (uint32_t)nd;
    }
    put(r + 8, (double)M[v]);
    put(r + 10, (double)C[v]);
    for (int sl = 0; sl < nd; ++sl) {
      const int i = dep_idx[dep_ptr[v] + sl];
      uint32_t* w = sl < 2 ? r + 2 + 2 * sl : r2 + 2 * (sl - 2);
      if (sl >= 2) r2[5 + (sl - 2)] = (uint32_t)i * 8u;
      uint32_t ref = kMNoFar;
      int nlate = 0;
      for (int32_t e = user_ptr[i]; e < user_ptr[i + 1]; ++e) {
        const int u = user_idx[e];
        if (u <= v) continue;
        if (u - v - 1 < 32) {
          w[0] |= 1u << (u - v - 1);
        } else {
          if (nlate++) return false;
          ref = far(u);
        }
      }
      w[1] = ref;
      put(sl < 2 ? r + 12 + 2 * sl : m23 + 2 * (sl - 2), (double)M[i]);
    }
    r[1] = ctrl;
    // the gate: below the stage's limit when a far reference may apply (the
    // low half takes node v-1's slot 1 offset below)
    r[7] = (ctrl & kMRare) ? 0u : std::min(ctrl, std::min(r[3], r[5])) & 0xFFFF0000u;
  }
  // fetch lists: record v (padded ones included) names the S_{t+1} words of
  // node v-1's slots 0 (word 6) and 1 (low half of word 7)
  for (int32_t v = 1; v < np; ++v) {
    const int32_t u = v - 1;
    uint32_t f0 = 0, f1 = 0;
    if (u < n) {
      const int nd = dep_ptr[u + 1] - dep_ptr[u];
      if (nd >= 1) f0 = (uint32_t)dep_idx[dep_ptr[u]] * 8u;
      if (nd >= 2) f1 = (uint32_t)dep_idx[dep_ptr[u] + 1] * 8u;
    }
    uint32_t* r = reinterpret_cast<uint32_t*>(base + (size_t)v * kMNodeBytes);
    r[6] = f0;
    r[7] = (r[7] & 0xFFFF0000u) | f1;
  }
  return true;   // node 0 keeps fetch list 0
}

bool build_seen_records(int32_t n, const int64_t* M, const int64_t* C, const int32_t* dep_ptr,
                        const int32_t* dep_idx, const int32_t* user_ptr, const int32_t* user_idx,
                        std::vector<char>& nodes, std::vector<uint32_t>& over, int32_t& seen_words,
                        int32_t tier_t[2], int32_t tier_w[2], int32_t& ntiers) {
  if (n < 1 || n > kSeenMaxNodes) return false;
  // seen bits: the nodes with a user more than 32 above them, in order of
  // their first such user (then of the node)
  std::vector<int32_t> first(n, INT32_MAX);
  std::vector<int32_t> order;
  for (int32_t x = 0; x < n; ++x) {
    for (int32_t e = user_ptr[x]; e < user_ptr[x + 1]; ++e)
      if (user_idx[e] - x - 1 >= 32) first[x] = std::min(first[x], user_idx[e]);
    if (first[x] != INT32_MAX) order.push_back(x);
  }
  std::stable_sort(order.begin(), order.end(), [&](int32_t x, int32_t y) { return first[x] < first[y]; });
  std::vector<int32_t> slot(n, -1);
  const int32_t ns = (int32_t)order.size();
  for (int32_t i = 0; i < ns; ++i) slot[order[i]] = i;
  seen_words = std::max<int32_t>(1, (ns + 31) / 32);
  // Stages t < T write only bits of nodes whose first far user is below T:
  // the first 32 w bits when T is the first far user of bit 32 w. Tiers at
  // three quarters and half of the words, where that is worth the launches
  // (at n = 4001, K = 4096: 76.4 ms per step against 79.3 with the half
  // alone and 90.7 with one launch; more tiers shorten the evaluate alone
  // but not the step, whose two streams each pay every launch boundary).
  ntiers = 0;
  if (seen_words >= kSeenSplitMinWords) {
    const int32_t ws[2] = {seen_words * 3 / 4, seen_words / 2};
    for (int i = 0; i < 2; ++i) {
      tier_t[ntiers] = first[order[32 * ws[i]]];
      tier_w[ntiers] = ws[i];
      ++ntiers;
    }
  }
  auto soff = [&](int32_t x) { return slot[x] < 0 ? 0u : (uint32_t)(slot[x] >> 5) * 256u; };
  auto sbit = [&](int32_t x) { return slot[x] < 0 ? 0u : 1u << (slot[x] & 31); };
  const int32_t np = n + 1;
  nodes.assign((size_t)np * kSNodeBytes, 0);
  over.clear();
  for (int32_t v = 0; v < n; ++v) {
    char* node = nodes.data() + (size_t)v * kSNodeBytes;
    uint32_t* r = reinterpret_cast<uint32_t*>(node);
    double* val = reinterpret_cast<double*>(node + 64);
    uint32_t* ext = reinterpret_cast<uint32_t*>(node + 112);
    for (int32_t e = user_ptr[v]; e < user_ptr[v + 1]; ++e) {
      const int32_t u = user_idx[e];
      if (u - v - 1 < 32) r[0] |= 1u << (u - v - 1);
    }
    r[1] = sbit(v);
    val[0] = (double)M[v];
    val[1] = (double)C[v];
    const int32_t nd = dep_ptr[v + 1] - dep_ptr[v];
    uint32_t flags = nd > 2 ? kSExt : 0u;
    if (nd > 4) {
      flags |= kSOver | (uint32_t)(nd - 4) << 8;
      r[8] = (uint32_t)(over.size() / 8);
    }
    r[2] = flags;
    for (int32_t sl = 0; sl < nd; ++sl) {
      const int32_t i = dep_idx[dep_ptr[v] + sl];
      uint32_t lm = 0;
      for (int32_t e = user_ptr[i]; e < user_ptr[i + 1]; ++e) {
        const int32_t u = user_idx[e];
        if (u > v && u - v - 1 < 32) lm |= 1u << (u - v - 1);
      }
      const uint32_t wr = v - i - 1 >= 32 ? (soff(i) | kSWrite) : 0u;
      if (sl < 2) {
        r[4 + 2 * sl] = lm;
        r[5 + 2 * sl] = sbit(i);
        r[3] |= wr << (16 * sl);
        val[2 + sl] = (double)M[i];
      } else if (sl < 4) {
        ext[2 * (sl - 2)] = lm;
        ext[2 * (sl - 2) + 1] = sbit(i);
        r[15] |= wr << (16 * (sl - 2));
        val[2 + sl] = (double)M[i];
      } else {
        const double mi = (double)M[i];
        uint32_t mw[2];
        memcpy(mw, &mi, sizeof(mw));
        const uint32_t en[8] = {lm, sbit(i), wr, (uint32_t)i * 8u, soff(i), mw[0], mw[1], 0u};
        over.insert(over.end(), en, en + 8);
      }
    }
  }
  // fetch blocks: node v's record describes node v-1's loads
  for (int32_t v = 1; v < np; ++v) {
    const int32_t u = v - 1;
    const int32_t nd = dep_ptr[u + 1] - dep_ptr[u];
    auto dep = [&](int32_t sl) { return dep_idx[dep_ptr[u] + sl]; };
    uint32_t* r = reinterpret_cast<uint32_t*>(nodes.data() + (size_t)v * kSNodeBytes);
    uint32_t f01 = 0, f23 = 0;
    if (nd >= 1) f01 |= (uint32_t)dep(0) * 8u;
    if (nd >= 2) f01 |= (uint32_t)dep(1) * 8u << 16;
    if (nd >= 3) {
      f01 |= kSExtNext;
      f23 |= (uint32_t)dep(2) * 8u;
    }
    if (nd >= 4) f23 |= (uint32_t)dep(3) * 8u << 16;
    r[9] = f01;
    r[10] = f23;
    r[11] = (uint32_t)u * (uint32_t)kSNodeBytes;
    r[12] = soff(u) | (nd >= 1 ? soff(dep(0)) : 0u) << 16;
    r[13] = (nd >= 2 ? soff(dep(1)) : 0u) | (nd >= 3 ? soff(dep(2)) : 0u) << 16;
    r[14] = nd >= 4 ? soff(dep(3)) : 0u;
  }
  return true;
}

void build_node_records(int32_t n, const int64_t* M, const int64_t* C, bool wide, const int32_t* dep_ptr,
                        const int32_t* dep_idx, const int32_t* user_ptr, const int32_t* user_idx,
                        void* out) {
  NodeRec* recs = static_cast<NodeRec*>(out);
  for (int32_t v = 0; v < n; ++v) {
    NodeRec r;
    memset(&r, 0, sizeof(r));
    r.M = rec_value(M[v], wide);
    r.C = rec_value(C[v], wide);
    // references, node n for "none": fu, then per slot s1 and fl
    int ref[1 + 2 * kRecDeps];
    for (int k = 0; k < 1 + 2 * kRecDeps; ++k) ref[k] = n;
    bool slow = false;
    int nfar = 0;
    for (int32_t e = user_ptr[v]; e < user_ptr[v + 1]; ++e) {
      const int u = user_idx[e];
      const int d = u - v - 1;
      if (d < 32) r.umask |= 1u << d;
      else if (nfar++ == 0) ref[0] = u;
    }
    if (nfar > 1) slow = true;
    const int nd = dep_ptr[v + 1] - dep_ptr[v];
    if (nd > kRecDeps) slow = true;
    for (int sl = 0; sl < nd && !slow; ++sl) {
      const int i = dep_idx[dep_ptr[v] + sl];
      ref[1 + 2 * sl] = i;
      r.dM[sl] = rec_value(M[i], wide);
      int nlate = 0;
      for (int32_t e = user_ptr[i]; e < user_ptr[i + 1]; ++e) {
        const int u = user_idx[e];
        if (u <= v) continue;
        const int d = u - v - 1;
        if (d < 32) r.lm[sl] |= 1u << d;
        else if (nlate++ == 0) ref[2 + 2 * sl] = u;
      }
      if (nlate > 1) slow = true;
    }
    const int ndeps = slow ? 0 : nd;
    // word indices (node >> 5 <= 128 fits 8 bits) and bit positions
    auto wd = [&](int k) { return (uint32_t)(ref[k] >> 5); };
    auto bp = [&](int k) { return (uint32_t)(ref[k] & 31); };
    r.refs0 = wd(0) | wd(2) << 8 | wd(1) << 16 | wd(4) << 24;
    r.refs1 = wd(3) | (uint32_t)ndeps << 8 | (slow ? kRefsSlow : 0u) | bp(6) << 12 | bp(7) << 17 | bp(8) << 22;
    r.refs2 = wd(6) | wd(5) << 8 | wd(8) << 16 | wd(7) << 24;
    for (int k = 0; k < 6; ++k) r.bits0 |= bp(k) << (5 * k);
    r.bits0 |= (slow ? 3u : (uint32_t)std::min(ndeps, 3)) << 30;
    r.mc[0] = r.M;
    r.mc[1] = r.C;
    r.dm01[0] = r.dM[0];
    r.dm01[1] = r.dM[1];
    if (slow) {
      // the slot fields are unused for a slow node: its lists go there
      // (kept only if they fit; the fields a slow node reads are untouched)
      uint32_t dw[64];
      memcpy(dw, &r, sizeof(dw));
      for (int k = 0; k < 64; ++k)
        if ((k < 4 || k >= 8) && (k < 24 || k >= 32)) dw[k] = 0;
      if (build_ext_lists(v, M, wide, dep_ptr, dep_idx, user_ptr, user_idx, dw)) memcpy(&r, dw, sizeof(dw));
    }
    recs[v] = r;
  }
}

}  // namespace ckm
