// Internal declarations shared by the host glue and the HIP kernels of libckm.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <mutex>
#include <vector>

#include "ckm.h"

namespace ckm {
struct SyncCache;  // buffers and stream of the synchronous entry points (ckm_host.cpp)
struct Fork;       // second stream of the overlapped producer/evaluate launches
}

// Graph on the device. Node arrays hold sizes and costs as int64. Users
// rows are sorted ascending; for the dep entry e = (i -> v) in v's deps row,
// dep_upos[e] is the index in user_idx of the first user of i that is
// greater than v. The evaluate kernels sum sizes and costs in binary64 when
// every sum they form stays below 2^53 (exact there), and in int64 otherwise
// (`wide`); the node records carry the values in the chosen form.
struct ckm_graph {
  int32_t n = 0;
  int32_t num_edges = 0;
  int device = 0;
  int64_t base = 0;           // M_in + 2 M_param (eq. U_init constant overhead)
  bool wide = false;          // sums reach 2^53: int64 arithmetic in the evaluate kernels
  int32_t eval_waves = 1;     // resident evaluate waves per CU for this n (work plan sizing)
  void* d_mem = nullptr;      // one allocation holding every array below
  const int64_t* d_M = nullptr;
  const int64_t* d_C = nullptr;
  const int32_t* d_user_ptr = nullptr;
  const int32_t* d_user_idx = nullptr;
  const int32_t* d_dep_ptr = nullptr;
  const int32_t* d_dep_idx = nullptr;
  const int32_t* d_dep_upos = nullptr;
  const void* d_recs = nullptr;  // n node records of ckm::kNodeRecBytes (see ckm_kernels.hip)
  const void* d_mrecs = nullptr; // mask-path records (mask_records_bytes) when the graph fits them, else NULL
  const void* d_snodes = nullptr; // else the seen path's node data, when the graph fits it
  const void* d_sover = nullptr;  // and its overflow entries (NULL when there are none)
  int32_t seen_words = 0;         // seen bits per lane / 32 on the seen path
  // seen-path launches by stage: the stages below seen_tier_t[i] touch only
  // the first seen_tier_w[i] words (seen_tiers of them, split stages falling)
  int32_t seen_tiers = 0;
  int32_t seen_tier_t[2] = {0, 0};
  int32_t seen_tier_w[2] = {0, 0};
  ckm::SyncCache* sync = nullptr;  // reused by the synchronous calls; freed with the graph
  ckm::Fork* fork = nullptr;       // NULL: every launch on the caller's stream
};

namespace ckm {

constexpr int kWave = 64;
constexpr int kNodeRecBytes = 256;
constexpr int kMaxNodesWords = CKM_MAX_NODES / 32;

// Where the evaluate kernel's S rows come from.
enum : int {
  kSrcRound = 0,      // randomized rounding of S* (deterministic candidate 0 under CKM_F_DET0)
  kSrcUser = 1,       // the caller's integral S matrices
  kSrcThreshold = 2,  // threshold rounding [clamp(S*) > p_k], one threshold per candidate
  kSrcRows = 3,       // randomized rounding done beforehand into the work buffer's row array
};

// The row arrays (S rows streamed by the evaluate kernel, R rows it keeps)
// are used when the S rows fit in this many bytes (about K * n^2 / 16 bytes
// each; 4.1 GB at n = 4001, K = 4096); larger problems, or work buffers sized
// without them, make the S rows in the evaluate kernel and recompute the best
// candidate's R.
constexpr size_t kRowsMaxBytes = (size_t)8 << 30;

// Host-side builder of the per-node records the evaluate kernel reads
// (layout documented with NodeRec in ckm_kernels.hip). Writes n records.
// M, C: int64 sizes and costs; wide: store them as int64 (else as binary64).
void build_node_records(int32_t n, const int64_t* M, const int64_t* C, bool wide, const int32_t* dep_ptr,
                        const int32_t* dep_idx, const int32_t* user_ptr, const int32_t* user_idx,
                        void* out);

// Records of the mask path (see ckm_kernels.hip), mask_records_bytes(n)
// of them; false when some node exceeds their format (more than four
// dependencies, more than one user more than 32 nodes above it, or a
// dependency with more than one such later user): the graph then takes the
// other kernels.
constexpr int kMaskPathMaxNodes = 1023;   // R row of up to 32 words in registers
int32_t mask_records_bytes(int32_t n);
bool build_mask_records(int32_t n, const int64_t* M, const int64_t* C, const int32_t* dep_ptr,
                        const int32_t* dep_idx, const int32_t* user_ptr, const int32_t* user_idx, void* out);
// Words of one candidate group's mask rows (rows 0 .. n).
size_t mask_rows_words(int32_t n);
// Node data of the seen path (see ckm_kernels.hip) for graphs of up to
// kSeenMaxNodes nodes: (n + 1) x 128 bytes, the overflow entries (8 dwords
// each) and the seen words per lane; false when n is too large. tier_t and
// tier_w (ntiers entries, at most 2): the stages below tier_t[i] touch only
// the first tier_w[i] seen words (no tiers where they would not pay).
constexpr int32_t kSeenMaxNodes = 4096;
bool build_seen_records(int32_t n, const int64_t* M, const int64_t* C, const int32_t* dep_ptr,
                        const int32_t* dep_idx, const int32_t* user_ptr, const int32_t* user_idx,
                        std::vector<char>& nodes, std::vector<uint32_t>& over, int32_t& seen_words,
                        int32_t tier_t[2], int32_t tier_w[2], int32_t& ntiers);
// Resident waves per CU of the mask and seen evaluate kernels.
int32_t mask_waves_per_cu();
int32_t seen_waves_per_cu(int32_t seen_words);

// Work-buffer layout for (n, K). Offsets are bytes from the buffer start,
// each 256-byte aligned.
struct Layout {
  int32_t n = 0, K = 0;
  int32_t ldq = 0;        // q / det row stride in elements: round_up(n + 8, 64)
  int32_t det_words = 0;  // ldq / 32
  int32_t row_words = 0;  // 32-bit words per output bit row: 2 * ceil(n / 64)
  int32_t max_splits = 0; // most work items per group of 64 candidates
  int32_t reduce_blocks = 0;
  // hdr: int32 number of work items (rows of the partial arrays) of the last evaluate
  size_t hdr_off = 0, q_off = 0, det_off = 0, nan_off = 0, part_peak_off = 0, part_cost_off = 0,
         best_off = 0, srows_off = 0, thr_sorted_off = 0, thr_rank_off = 0,
         // execution plans: per-stage statement and compute counts, check
         // flags, first statement and first register, and the go flag
         plan_cnt_off = 0, plan_comp_off = 0, plan_err_off = 0, plan_pos_off = 0, plan_rbase_off = 0,
         plan_go_off = 0,
         // R transposed (n columns of ceil(n/32) words) and per-row word ranks
         plan_rt_off = 0, plan_rpre_off = 0,
         bbest_off = 0,  // per-block best of the batch multipliers
         total = 0,        // bytes every call needs
         rows_off = 0,     // S rows of every candidate (kSrcRows), past `total`
         rrows_off = 0,    // R rows of every candidate, written by the evaluate stage
         total_rows = 0;   // total plus the two row arrays when they are used
  bool rows_on = false;    // the S rows fit kRowsMaxBytes (and, after
                           // check_work, the caller's buffer holds both arrays)
};

Layout make_layout(int32_t n, int32_t K);

// Records a thread-local error message (ckm_last_error) and returns st.
ckm_status set_error(ckm_status st, const char* fmt, ...);

// The static work area of ckm_round_eval_noalloc (ckm_noalloc.hip):
// noalloc_setup resolves its address on `device`, which must be current
// (graph creation calls it); noalloc_scratch returns the kept address, or
// NULL when the device was never set up.
hipError_t noalloc_setup(int device);
void* noalloc_scratch(int device);

// How the stages of one group of 64 candidates are cut into work items (one
// wave each). Items are numbered in dispatch order, most expensive first, so
// the cheap ones fill the end of the launch.
//   kind 0: `items` ranges of about equal sum of stage lengths, top first.
//   kind 1: stages T0 .. n-1 in R1 items of P consecutive stages (top
//           first), then stages 0 .. T0-1 in R2 ranges of about equal sum of
//           stage lengths (top first).
struct Plan {
  int32_t items = 1, kind = 0, P = 0, T0 = 0, R1 = 0, R2 = 0;
};
Plan plan_auto(int32_t n, int32_t K, int32_t max_items, int32_t waves_per_cu);
Plan plan_stages(int32_t n, int32_t max_items);
Plan plan_splits(int32_t n, int32_t splits);

// Resident evaluate waves per CU for a graph of n nodes (the runtime's
// occupancy figure for the kernel variant and LDS size n and wide select).
int32_t eval_waves_per_cu(int32_t n, bool wide);

// A second stream and two events, made with a seen-path graph on its device,
// over which launch_evaluate splits its candidate groups in two chunks: the
// second chunk's producer and evaluate run beside the first chunk's evaluate.
// The mutex keeps one call's record/wait sequence on the events whole.
struct Fork {
  std::mutex mu;
  hipStream_t side = nullptr;
  hipEvent_t forked = nullptr, joined = nullptr;
};
// Seen-path evaluates resident at no more than this many waves per CU (held
// there by their LDS) get the overlapped launch and so the second stream.
constexpr int32_t kForkMaxWaves = 16;
hipError_t fork_create(Fork& f);
void fork_destroy(Fork& f);

// ckm_round_eval_async, with the overlapped launch on or off (off for the
// entry point that creates and allocates nothing).
ckm_status round_eval(const ckm_graph* g, const double* d_s_frac, int64_t ld, int32_t K, uint64_t seed,
                      int64_t budget, uint32_t flags, int64_t* d_peak, int64_t* d_cost, uint8_t* d_feasible,
                      int32_t* d_best_k, uint64_t* d_best_S, uint64_t* d_best_R, int32_t* d_status, void* d_work,
                      size_t work_bytes, void* stream, bool overlap);

// Kernel launchers (defined in ckm_kernels.hip). They only enqueue work.
hipError_t launch_quantize(const ckm_graph& g, const Layout& L, const double* d_s, int64_t ld,
                           char* work, hipStream_t stream);
// Randomized path: every candidate's S rows rounded once into the work
// buffer's row array (nothing when L.rows_on is false).
hipError_t launch_round_rows(const ckm_graph& g, const Layout& L, int32_t K, uint64_t seed, uint32_t flags,
                             char* work, hipStream_t stream);
// The same for candidate groups g0 .. g0 + gn - 1 (64 candidates each);
// clear: on the mask path, also reset those candidates' evaluate totals.
hipError_t launch_round_rows(const ckm_graph& g, const Layout& L, int32_t K, uint64_t seed, uint32_t flags,
                             int32_t g0, int32_t gn, bool clear, char* work, hipStream_t stream);
// Threshold family: ranks of the K thresholds, their sorted copy, and the
// keys of S* in place of the quantized thresholds q.
hipError_t launch_threshold_keys(const ckm_graph& g, const Layout& L, const double* d_s, int64_t ld,
                                 const double* d_p, int32_t K, char* work, hipStream_t stream);
// Execution plan of (S, R) (bit rows of row_words 32-bit words): counts,
// checks and prefix sums, then the statements when d_P is not null.
hipError_t launch_plan(const ckm_graph& g, const Layout& L, const uint64_t* d_S, const uint64_t* d_R,
                       uint32_t flags, int32_t* d_P, int64_t capacity, int64_t* d_count, int64_t* d_mem,
                       int32_t* d_status, char* work, hipStream_t stream);
// Largest batch multiplier per candidate from the totals of the last
// evaluate, and the best one.
hipError_t launch_max_batch(const ckm_graph& g, const Layout& L, int32_t K, int64_t budget, int64_t cost_cap,
                            int64_t* d_batch, int32_t* d_best_k, int64_t* d_best_batch, int32_t* d_status,
                            char* work, hipStream_t stream);
// src: one of kSrcRound, kSrcUser, kSrcThreshold (kSrcRound streams the row
// array when L.rows_on, rounding it first unless flags has CKM_F_ROUNDED).
// s_user: for kSrcUser, K
// caller-supplied S matrices ([K][n][row_words] 32-bit words).
// With overlap, the candidate groups are split over the caller's stream and
// g.fork's (when the graph has one and K is large enough); the caller's
// stream waits for the other before it returns, as after one launch.
hipError_t launch_evaluate(const ckm_graph& g, const Layout& L, int32_t K, uint64_t seed,
                           uint32_t flags, const Plan& plan, int src, const uint64_t* s_user, char* work,
                           hipStream_t stream, bool overlap = true);
hipError_t launch_select(const ckm_graph& g, const Layout& L, int32_t K, uint64_t seed,
                         int64_t budget, uint32_t flags, int64_t* d_peak,
                         int64_t* d_cost, uint8_t* d_feasible, int32_t* d_best_k,
                         uint64_t* d_best_S, uint64_t* d_best_R, int32_t* d_status, int src,
                         const uint64_t* s_user, char* work, hipStream_t stream);

}  // namespace ckm
