// Host side of libckm: argument and graph validation, device upload, the
// work-buffer layout and the C ABI entry points declared in include/ckm.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "ckm_internal.h"

namespace {

thread_local std::string g_last_error;

ckm_status fail(ckm_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

ckm_status fail_hip(hipError_t e, const char* what) {
  return fail(CKM_E_DEVICE, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

constexpr int64_t kExactLimit = int64_t(1) << 53;  // binary64 integers are exact below this

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Restores the caller's current device on scope exit.
struct DeviceGuard {
  int prev = -1;
  bool ok = false;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) return;
    ok = (prev == dev) || (hipSetDevice(dev) == hipSuccess);
  }
  ~DeviceGuard() {
    if (ok && prev >= 0) (void)hipSetDevice(prev);
  }
};

}  // namespace

namespace ckm {

ckm_status set_error(ckm_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

// Device memory, pinned host memory and a stream for the synchronous entry
// points, kept on the graph so that repeated calls allocate nothing after the
// first. The buffers grow to the largest call seen and are released with the
// graph.
struct SyncCache {
  std::mutex mu;
  hipStream_t stream = nullptr;
  char* d = nullptr;
  size_t d_bytes = 0;
  char* h = nullptr;
  size_t h_bytes = 0;

  // Waits for queued work, then frees everything (the graph's device is current).
  void release() {
    if (stream) {
      (void)hipStreamSynchronize(stream);
      (void)hipStreamDestroy(stream);
      stream = nullptr;
    }
    if (d) (void)hipFree(d);
    if (h) (void)hipHostFree(h);
    d = h = nullptr;
    d_bytes = h_bytes = 0;
  }
};

}  // namespace ckm

namespace {

// One synchronous call's hold on the graph's SyncCache. When another thread
// holds the cache, the call uses private buffers freed at its end, so
// synchronous calls on a shared graph remain safe to run concurrently. The
// destructor waits for the stream; construct after the DeviceGuard.
class SyncCall {
 public:
  explicit SyncCall(const ckm_graph* g) : lk_(g->sync->mu, std::try_to_lock) {
    c_ = lk_.owns_lock() ? g->sync : &own_;
  }
  ~SyncCall() {
    if (c_ == &own_) {
      own_.release();
    } else if (c_->stream) {
      (void)hipStreamSynchronize(c_->stream);
    }
  }
  SyncCall(const SyncCall&) = delete;
  SyncCall& operator=(const SyncCall&) = delete;

  // At least d_bytes of device memory and h_bytes of pinned host memory.
  ckm_status reserve(size_t d_bytes, size_t h_bytes) {
    hipError_t e;
    if (!c_->stream && (e = hipStreamCreateWithFlags(&c_->stream, hipStreamNonBlocking)) != hipSuccess) {
      c_->stream = nullptr;
      return fail_hip(e, "hipStreamCreate");
    }
    // the shared buffers are rounded up to 2 MiB, so that slightly larger
    // calls reuse them
    constexpr size_t kStep = (size_t)2 << 20;
    const bool shared = c_ != &own_;
    auto grow = [&](size_t need) { return shared ? (need + kStep - 1) / kStep * kStep : need; };
    if (d_bytes > c_->d_bytes) {
      (void)hipStreamSynchronize(c_->stream);
      if (c_->d) (void)hipFree(c_->d);
      c_->d = nullptr;
      c_->d_bytes = 0;
      const size_t sz = grow(d_bytes);
      if ((e = hipMalloc(&c_->d, sz)) != hipSuccess) {
        c_->d = nullptr;
        return e == hipErrorOutOfMemory ? fail(CKM_E_NOMEM, "hipMalloc of %zu bytes failed", sz)
                                        : fail_hip(e, "hipMalloc");
      }
      c_->d_bytes = sz;
    }
    if (h_bytes > c_->h_bytes) {
      (void)hipStreamSynchronize(c_->stream);
      if (c_->h) (void)hipHostFree(c_->h);
      c_->h = nullptr;
      c_->h_bytes = 0;
      const size_t sz = grow(h_bytes);
      if ((e = hipHostMalloc(reinterpret_cast<void**>(&c_->h), sz, hipHostMallocDefault)) != hipSuccess) {
        c_->h = nullptr;
        return e == hipErrorOutOfMemory ? fail(CKM_E_NOMEM, "hipHostMalloc of %zu bytes failed", sz)
                                        : fail_hip(e, "hipHostMalloc");
      }
      c_->h_bytes = sz;
    }
    return CKM_OK;
  }

  hipStream_t stream() const { return c_->stream; }
  char* dev() const { return c_->d; }
  char* host() const { return c_->h; }

  // Waits for the stream; maps a failure to CKM_E_DEVICE.
  ckm_status wait() {
    const hipError_t e = hipStreamSynchronize(c_->stream);
    return e == hipSuccess ? CKM_OK : fail_hip(e, "hipStreamSynchronize");
  }

 private:
  std::unique_lock<std::mutex> lk_;
  ckm::SyncCache own_;
  ckm::SyncCache* c_ = nullptr;
};

// Copies the strict lower triangle of S* (n rows of stride ld) into the
// pinned buffer h as an n x n row-major matrix and uploads it to d in blocks
// of rows, each block's upload overlapping the copy of the next. Entries on
// and above the diagonal are neither read nor copied (the kernels never read
// them). A NaN in the lower triangle is an error.
ckm_status stage_s_frac(const double* s, int64_t ld, int32_t n, double* h, char* d, hipStream_t stream) {
  const int32_t block = std::max<int32_t>(1, (1 << 17) / std::max(n, 1));  // about 1 MiB of rows
  for (int32_t t0 = 0; t0 < n; t0 += block) {
    const int32_t t1 = std::min(n, t0 + block);
    for (int32_t t = t0; t < t1; ++t) {
      const double* src = s + (int64_t)t * ld;
      double* dst = h + (int64_t)t * n;
      bool bad = false;
      for (int32_t i = 0; i < t; ++i) {
        const double x = src[i];
        bad |= std::isnan(x);
        dst[i] = x;
      }
      if (bad) {
        for (int32_t i = 0; i < t; ++i)
          if (std::isnan(src[i])) return fail(CKM_E_INVALID_ARG, "S*[%d][%d] is NaN", t, i);
      }
    }
    const size_t off = (size_t)t0 * n * sizeof(double);
    const hipError_t e = hipMemcpyAsync(d + off, reinterpret_cast<char*>(h) + off,
                                        (size_t)(t1 - t0) * n * sizeof(double), hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return fail_hip(e, "hipMemcpy S*");
  }
  return CKM_OK;
}

// A result array copied from the device buffer (at off) to the caller.
struct Result {
  void* dst;
  size_t off, bytes;
};

// Downloads the device range [lo, hi) that holds every result in one copy
// into the pinned buffer at h_off, waits, and hands each result on.
ckm_status fetch_results(SyncCall& sc, size_t lo, size_t hi, size_t h_off, const Result* r, int count) {
  hipError_t e = hipMemcpyAsync(sc.host() + h_off, sc.dev() + lo, hi - lo, hipMemcpyDeviceToHost, sc.stream());
  if (e != hipSuccess) return fail_hip(e, "hipMemcpy results");
  const ckm_status st = sc.wait();
  if (st != CKM_OK) return st;
  for (int i = 0; i < count; ++i)
    if (r[i].dst) memcpy(r[i].dst, sc.host() + h_off + (r[i].off - lo), r[i].bytes);
  return CKM_OK;
}

}  // namespace

namespace ckm {

int32_t max_splits_for(int32_t n, int32_t /*K*/) {
  // work items per group of 64 candidates: at most one per stage
  return std::max<int32_t>(n, 1);
}

Plan plan_splits(int32_t n, int32_t splits) {
  Plan p;
  p.kind = 0;
  p.items = std::max(1, std::min(splits, n));
  return p;
}

Plan plan_auto(int32_t n, int32_t K, int32_t max_items, int32_t waves_per_cu) {
  // About eight items per resident wave slot. Stages from T0 = n/16 up go in
  // items of P stages (one stage when there are enough items), the first
  // n/16 stages in as many small ranges, so the launch, which dispatches
  // the most expensive items first, ends on very short ones. Each item
  // regenerates one S row; the shorter tail is worth more than that (at
  // n = 1009, K = 1024: 0.94 ms against 1.00 with T0 = n/2).
  const int64_t groups = (K + kWave - 1) / kWave;
  // resident evaluate waves on the chip's 256 CUs
  const int64_t slots = 256 * (int64_t)std::max(1, waves_per_cu);
  const int64_t target = std::max<int64_t>(1, (8 * slots + groups - 1) / groups);
  if (n < 8 || target < 4) return plan_splits(n, (int32_t)std::min<int64_t>(target, max_items));
  Plan p;
  p.kind = 1;
  p.T0 = std::max(1, n / 16);
  const int64_t half = std::max<int64_t>(1, target / 2);
  p.P = (int32_t)std::max<int64_t>(1, (n - p.T0 + half - 1) / half);
  for (;;) {
    p.R1 = (n - p.T0 + p.P - 1) / p.P;
    p.R2 = std::max(1, std::min(p.T0, p.R1));
    p.items = p.R1 + p.R2;
    if (p.items <= max_items || p.P >= n) break;
    p.P *= 2;
  }
  if (p.items > max_items) return plan_splits(n, max_items);
  return p;
}

Plan plan_stages(int32_t n, int32_t max_items) {
  // One stage per item from T0 = n/16 up, the longest first, then the first
  // T0 stages in T0 items: the mask and seen kernels read each stage's rows
  // from the row array, so an item costs no more than its stages, and the
  // finest items balance best (n = 4001, K = 4096: 89 ms per evaluate
  // against 93 with the 24-stage items of plan_auto).
  if (n < 8) return plan_splits(n, max_items);
  Plan p;
  p.kind = 1;
  p.T0 = std::max(1, n / 16);
  p.P = 1;
  p.R1 = n - p.T0;
  p.R2 = std::max(1, std::min(p.T0, p.R1));
  p.items = p.R1 + p.R2;
  if (p.items > max_items) return plan_splits(n, max_items);
  return p;
}

// The automatic plan of a graph's evaluate: one stage per item on the mask
// and seen kernels (they need the row arrays), plan_auto otherwise.
static Plan plan_for(const ckm_graph* g, const Layout& L, int32_t K) {
  if (L.rows_on && (g->d_mrecs || g->d_snodes)) return plan_stages(g->n, L.max_splits);
  return plan_auto(g->n, K, L.max_splits, g->eval_waves);
}

Layout make_layout(int32_t n, int32_t K) {
  Layout L;
  L.n = n;
  L.K = K;
  L.ldq = ((n + 8 + 63) / 64) * 64;
  L.det_words = L.ldq / 32;
  L.row_words = 2 * ((n + 63) / 64);
  L.max_splits = max_splits_for(n, K);
  L.reduce_blocks = (K + 255) / 256;
  size_t off = 0;
  L.hdr_off = off;       off = align256(off + 256);
  L.q_off = off;         off = align256(off + (size_t)n * L.ldq * sizeof(uint32_t));
  L.det_off = off;       off = align256(off + (size_t)n * L.det_words * sizeof(uint32_t));
  L.nan_off = off;       off = align256(off + (size_t)n * sizeof(int32_t));
  L.part_peak_off = off; off = align256(off + (size_t)K * sizeof(int64_t));
  L.part_cost_off = off; off = align256(off + (size_t)K * sizeof(int64_t));
  L.best_off = off;      off = align256(off + (size_t)L.reduce_blocks * 24);
  L.srows_off = off;     off = align256(off + (size_t)n * L.row_words * sizeof(uint32_t));
  // threshold family: sorted thresholds and per-candidate ranks
  const size_t kt = (size_t)std::min<int32_t>(K, CKM_MAX_THRESHOLDS);
  L.thr_sorted_off = off; off = align256(off + kt * sizeof(double));
  L.thr_rank_off = off;   off = align256(off + kt * sizeof(uint32_t));
  L.plan_cnt_off = off;   off = align256(off + (size_t)n * sizeof(int64_t));
  L.plan_comp_off = off;  off = align256(off + (size_t)n * sizeof(int64_t));
  L.plan_err_off = off;   off = align256(off + (size_t)n * sizeof(int32_t));
  L.plan_pos_off = off;   off = align256(off + (size_t)n * sizeof(int64_t));
  L.plan_rbase_off = off; off = align256(off + (size_t)n * sizeof(int64_t));
  L.plan_go_off = off;    off = align256(off + sizeof(int32_t));
  L.plan_rt_off = off;    off = align256(off + (size_t)n * ((n + 31) / 32) * sizeof(uint32_t));
  L.plan_rpre_off = off;  off = align256(off + (size_t)n * ckm::kMaxNodesWords * sizeof(int32_t));
  L.bbest_off = off;      off = align256(off + (size_t)L.reduce_blocks * 32);

  L.total = off;
  // S rows, then R rows, of every candidate, word w of row t at
  // (base(t) + w) * kpad + k: last, and optional (without them the evaluate
  // stage makes its S rows itself and select recomputes the best R)
  const size_t kpad = (size_t)((K + kWave - 1) / kWave) * kWave;
  const size_t full = (size_t)(n >> 5), rem = (size_t)(n & 31);
  const size_t rrows_bytes = kpad * (32 * full * (full + 1) / 2 + rem * (full + 1)) * sizeof(uint32_t);
  // the S rows are in this layout, or (the mask path) as one 64-bit word per
  // group of 64 candidates and node: room for the larger of the two
  const size_t mask_bytes = (kpad / kWave) * ckm::mask_rows_words(n) * sizeof(uint64_t);
  const size_t rows_bytes = std::max(rrows_bytes, mask_bytes);
  L.rows_on = rows_bytes <= ckm::kRowsMaxBytes;
  L.rows_off = off;
  L.rrows_off = align256(off + rows_bytes);
  L.total_rows = L.rows_on ? align256(L.rrows_off + rrows_bytes) : off;
  return L;
}

}  // namespace ckm

using ckm::Layout;

extern "C" {

const char* ckm_last_error(void) { return g_last_error.c_str(); }

int32_t ckm_graph_num_nodes(const ckm_graph* g) { return g ? g->n : -1; }

static ckm_status graph_create(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                               const int32_t* user_ptr, const int32_t* user_idx, const int64_t* cost,
                               const int64_t* bytes, int64_t m_input, int64_t m_param, ckm_graph** out);

ckm_status ckm_graph_create(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                            const int32_t* user_ptr, const int32_t* user_idx,
                            const int64_t* cost, const int64_t* bytes, int64_t m_input,
                            int64_t m_param, ckm_graph** out) {
  if (!out) return fail(CKM_E_INVALID_ARG, "out is NULL");
  *out = nullptr;
  // the host-side vectors are the only allocations here that throw
  try {
    return graph_create(n, dep_ptr, dep_idx, user_ptr, user_idx, cost, bytes, m_input, m_param, out);
  } catch (const std::bad_alloc&) {
    return fail(CKM_E_NOMEM, "out of host memory");
  }
}

static ckm_status graph_create(int32_t n, const int32_t* dep_ptr, const int32_t* dep_idx,
                               const int32_t* user_ptr, const int32_t* user_idx, const int64_t* cost,
                               const int64_t* bytes, int64_t m_input, int64_t m_param, ckm_graph** out) {
  if (n < 1) return fail(CKM_E_INVALID_ARG, "n = %d < 1", n);
  if (n > CKM_MAX_NODES) return fail(CKM_E_UNSUPPORTED, "n = %d > %d", n, CKM_MAX_NODES);
  if (!dep_ptr || !cost || !bytes) return fail(CKM_E_INVALID_ARG, "NULL dep_ptr, cost or bytes");
  if (!user_ptr && user_idx)
    return fail(CKM_E_INVALID_ARG, "user_idx given without user_ptr");
  if (dep_ptr[0] != 0) return fail(CKM_E_GRAPH, "dep_ptr[0] = %d, expected 0", dep_ptr[0]);
  for (int32_t j = 0; j < n; ++j)
    if (dep_ptr[j + 1] < dep_ptr[j]) return fail(CKM_E_GRAPH, "dep_ptr decreases at %d", j);
  const int32_t E = dep_ptr[n];
  // edges i -> j with i < j, no two alike: at most n (n - 1) / 2 of them
  if ((int64_t)E > (int64_t)n * (n - 1) / 2)
    return fail(CKM_E_GRAPH, "%d edges on %d nodes: some edge repeats or is not in topological order", E, n);
  if (E > 0 && !dep_idx) return fail(CKM_E_INVALID_ARG, "dep_idx is NULL with %d edges", E);
  if (m_input < 0 || m_param < 0) return fail(CKM_E_INVALID_ARG, "negative m_input or m_param");

  // Deps rows: in range, topological (i < j), no duplicates; stored sorted.
  std::vector<int32_t> dp(dep_ptr, dep_ptr + n + 1), di(E);
  std::vector<int32_t> seen(n, -1);
  for (int32_t j = 0; j < n; ++j) {
    for (int32_t a = dep_ptr[j]; a < dep_ptr[j + 1]; ++a) {
      const int32_t i = dep_idx[a];
      if (i < 0 || i >= j)
        return fail(CKM_E_GRAPH, "edge %d -> %d is not in topological order", i, j);
      if (seen[i] == j) return fail(CKM_E_GRAPH, "duplicate edge %d -> %d", i, j);
      seen[i] = j;
      di[a] = i;
    }
    std::sort(di.begin() + dp[j], di.begin() + dp[j + 1]);
  }
  // Sizes and costs: non-negative; M_in + 2 M_param + sum(M) and n sum(C)
  // within int64 (every memory level and every cost the method forms is at
  // most these).
  int64_t total_m = m_input, total_c = 0;
  auto add_checked = [](int64_t& acc, int64_t v) {
    if (v > INT64_MAX - acc) return false;
    acc += v;
    return true;
  };
  if (!add_checked(total_m, m_param) || !add_checked(total_m, m_param))
    return fail(CKM_E_OVERFLOW, "M_in + 2 M_param exceeds INT64_MAX");
  for (int32_t v = 0; v < n; ++v) {
    if (cost[v] < 0 || bytes[v] < 0)
      return fail(CKM_E_INVALID_ARG, "negative cost or size at node %d", v);
    if (!add_checked(total_m, bytes[v]))
      return fail(CKM_E_OVERFLOW, "M_in + 2 M_param + sum(M) exceeds INT64_MAX");
    if (!add_checked(total_c, cost[v])) return fail(CKM_E_OVERFLOW, "sum(C) exceeds INT64_MAX");
  }
  if (total_c > 0 && (int64_t)n > INT64_MAX / total_c)
    return fail(CKM_E_OVERFLOW, "n * sum(C) exceeds INT64_MAX");
  // binary64 sums are exact while every partial sum stays below 2^53: each
  // stage's memory levels are at most M_in + 2 M_param + sum(M), its cost at
  // most sum(C) (the stage costs are added in int64)
  const bool wide = total_m >= kExactLimit || total_c >= kExactLimit;

  // Users = transpose(Deps), rows ascending.
  std::vector<int32_t> up(n + 1, 0), ui(E);
  for (int32_t a = 0; a < E; ++a) up[di[a] + 1]++;
  for (int32_t i = 0; i < n; ++i) up[i + 1] += up[i];
  {
    std::vector<int32_t> fill(up.begin(), up.end() - 1);
    for (int32_t j = 0; j < n; ++j)
      for (int32_t a = dp[j]; a < dp[j + 1]; ++a) ui[fill[di[a]]++] = j;  // j ascending
  }
  if (user_ptr) {
    if (E > 0 && !user_idx) return fail(CKM_E_INVALID_ARG, "user_idx is NULL with %d edges", E);
    if (user_ptr[0] != 0 || user_ptr[n] != E)
      return fail(CKM_E_GRAPH, "users CSR does not have the edge count of deps");
    for (int32_t i = 0; i < n; ++i)
      if (user_ptr[i + 1] < user_ptr[i]) return fail(CKM_E_GRAPH, "user_ptr decreases at %d", i);
    for (int32_t i = 0; i < n; ++i) {
      if (user_ptr[i + 1] - user_ptr[i] != up[i + 1] - up[i])
        return fail(CKM_E_GRAPH, "users of node %d differ from the transpose of deps", i);
      std::vector<int32_t> got(user_idx + user_ptr[i], user_idx + user_ptr[i + 1]);
      std::sort(got.begin(), got.end());
      if (!std::equal(got.begin(), got.end(), ui.begin() + up[i]))
        return fail(CKM_E_GRAPH, "users of node %d differ from the transpose of deps", i);
    }
  }
  // dep_upos: for entry (i -> j), first position in Users[i] after j.
  std::vector<int32_t> upos(E);
  for (int32_t j = 0; j < n; ++j)
    for (int32_t a = dp[j]; a < dp[j + 1]; ++a) {
      const int32_t i = di[a];
      const int32_t* b = ui.data() + up[i];
      const int32_t* e = ui.data() + up[i + 1];
      upos[a] = (int32_t)(std::upper_bound(b, e, j) - ui.data());
    }

  const size_t Ea = (size_t)std::max(E, 1);
  const size_t off_M = 0;
  const size_t off_C = align256(off_M + n * sizeof(int64_t));
  const size_t off_up = align256(off_C + n * sizeof(int64_t));
  const size_t off_ui = align256(off_up + (n + 1) * sizeof(int32_t));
  const size_t off_dp = align256(off_ui + Ea * sizeof(int32_t));
  const size_t off_di = align256(off_dp + (n + 1) * sizeof(int32_t));
  const size_t off_uo = align256(off_di + Ea * sizeof(int32_t));
  const size_t off_rec = align256(off_uo + Ea * sizeof(int32_t));
  const size_t off_mrec = align256(off_rec + (size_t)n * ckm::kNodeRecBytes);
  // the mask path's records, when the graph fits their format
  std::vector<char> mrecs;
  if (!wide && n <= ckm::kMaskPathMaxNodes) {
    mrecs.resize((size_t)ckm::mask_records_bytes(n));
    if (!ckm::build_mask_records(n, bytes, cost, dp.data(), di.data(), up.data(), ui.data(), mrecs.data()))
      mrecs.clear();
  }
  // else the seen path's node data, when the graph fits it
  std::vector<char> snodes;
  std::vector<uint32_t> sover;
  int32_t seen_words = 0, seen_tiers = 0, seen_tier_t[2] = {0, 0}, seen_tier_w[2] = {0, 0};
  if (mrecs.empty() && !wide &&
      !ckm::build_seen_records(n, bytes, cost, dp.data(), di.data(), up.data(), ui.data(), snodes, sover,
                               seen_words, seen_tier_t, seen_tier_w, seen_tiers))
    snodes.clear();
  const size_t off_snode = align256(off_mrec + mrecs.size());
  const size_t off_sover = align256(off_snode + snodes.size());
  const size_t total = align256(off_sover + sover.size() * sizeof(uint32_t));
  std::vector<char> host(total, 0);
  if (!mrecs.empty()) memcpy(host.data() + off_mrec, mrecs.data(), mrecs.size());
  if (!snodes.empty()) memcpy(host.data() + off_snode, snodes.data(), snodes.size());
  if (!sover.empty()) memcpy(host.data() + off_sover, sover.data(), sover.size() * sizeof(uint32_t));
  memcpy(host.data() + off_M, bytes, n * sizeof(int64_t));
  memcpy(host.data() + off_C, cost, n * sizeof(int64_t));
  memcpy(host.data() + off_up, up.data(), (n + 1) * sizeof(int32_t));
  if (E) memcpy(host.data() + off_ui, ui.data(), E * sizeof(int32_t));
  memcpy(host.data() + off_dp, dp.data(), (n + 1) * sizeof(int32_t));
  if (E) memcpy(host.data() + off_di, di.data(), E * sizeof(int32_t));
  if (E) memcpy(host.data() + off_uo, upos.data(), E * sizeof(int32_t));
  ckm::build_node_records(n, bytes, cost, wide, dp.data(), di.data(), up.data(), ui.data(),
                          host.data() + off_rec);

  ckm_graph* g = new (std::nothrow) ckm_graph();
  if (!g) return fail(CKM_E_NOMEM, "host allocation failed");
  g->n = n;
  g->num_edges = E;
  g->base = m_input + 2 * m_param;
  g->wide = wide;
  hipError_t e = hipGetDevice(&g->device);
  if (e != hipSuccess) {
    delete g;
    return fail_hip(e, "hipGetDevice");
  }
  g->eval_waves = !mrecs.empty()    ? ckm::mask_waves_per_cu()
                  : !snodes.empty() ? ckm::seen_waves_per_cu(seen_words)
                                    : ckm::eval_waves_per_cu(n, wide);
  // the work area of ckm_round_eval_noalloc on this device, resolved once
  e = ckm::noalloc_setup(g->device);
  if (e != hipSuccess) {
    delete g;
    return fail_hip(e, "resolving the no-allocation work area");
  }
  e = hipMalloc(&g->d_mem, total);
  if (e != hipSuccess) {
    delete g;
    return e == hipErrorOutOfMemory ? fail(CKM_E_NOMEM, "hipMalloc of %zu bytes failed", total)
                                    : fail_hip(e, "hipMalloc");
  }
  e = hipMemcpy(g->d_mem, host.data(), total, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(g->d_mem);
    delete g;
    return fail_hip(e, "hipMemcpy graph upload");
  }
  char* base = static_cast<char*>(g->d_mem);
  g->d_M = reinterpret_cast<const int64_t*>(base + off_M);
  g->d_C = reinterpret_cast<const int64_t*>(base + off_C);
  g->d_user_ptr = reinterpret_cast<const int32_t*>(base + off_up);
  g->d_user_idx = reinterpret_cast<const int32_t*>(base + off_ui);
  g->d_dep_ptr = reinterpret_cast<const int32_t*>(base + off_dp);
  g->d_dep_idx = reinterpret_cast<const int32_t*>(base + off_di);
  g->d_dep_upos = reinterpret_cast<const int32_t*>(base + off_uo);
  g->d_recs = base + off_rec;
  g->d_mrecs = mrecs.empty() ? nullptr : base + off_mrec;
  g->d_snodes = snodes.empty() ? nullptr : base + off_snode;
  g->d_sover = snodes.empty() || sover.empty() ? nullptr : base + off_sover;
  g->seen_words = seen_words;
  g->seen_tiers = seen_tiers;
  for (int i = 0; i < 2; ++i) {
    g->seen_tier_t[i] = seen_tier_t[i];
    g->seen_tier_w[i] = seen_tier_w[i];
  }
  g->sync = new (std::nothrow) ckm::SyncCache;
  if (!g->sync) {
    (void)hipFree(g->d_mem);
    delete g;
    return fail(CKM_E_NOMEM, "out of host memory");
  }
  // the side stream of the overlapped launches (seen-path graphs whose
  // evaluate LDS holds to a few waves per SIMD)
  if (g->d_snodes && g->eval_waves <= ckm::kForkMaxWaves) {
    g->fork = new (std::nothrow) ckm::Fork;
    e = g->fork ? ckm::fork_create(*g->fork) : hipErrorOutOfMemory;
    if (e != hipSuccess) {
      delete g->fork;
      g->sync->release();
      delete g->sync;
      (void)hipFree(g->d_mem);
      delete g;
      return fail_hip(e, "side stream");
    }
  }
  *out = g;
  return CKM_OK;
}

void ckm_graph_destroy(ckm_graph* g) {
  if (!g) return;
  DeviceGuard dg(g->device);
  if (g->fork) {
    ckm::fork_destroy(*g->fork);
    delete g->fork;
  }
  if (g->sync) {
    g->sync->release();
    delete g->sync;
  }
  if (g->d_mem) (void)hipFree(g->d_mem);
  delete g;
}

ckm_status ckm_workspace_size(const ckm_graph* g, int32_t K, size_t* bytes) {
  if (!g || !bytes) return fail(CKM_E_INVALID_ARG, "NULL graph or bytes");
  if (K < 1) return fail(CKM_E_INVALID_ARG, "K = %d < 1", K);
  if (K > CKM_MAX_CANDIDATES) return fail(CKM_E_UNSUPPORTED, "K = %d > %d", K, CKM_MAX_CANDIDATES);
  *bytes = ckm::make_layout(g->n, K).total_rows;
  return CKM_OK;
}

ckm_status ckm_workspace_size_min(const ckm_graph* g, int32_t K, size_t* bytes) {
  if (!g || !bytes) return fail(CKM_E_INVALID_ARG, "NULL graph or bytes");
  if (K < 1) return fail(CKM_E_INVALID_ARG, "K = %d < 1", K);
  if (K > CKM_MAX_CANDIDATES) return fail(CKM_E_UNSUPPORTED, "K = %d > %d", K, CKM_MAX_CANDIDATES);
  *bytes = ckm::make_layout(g->n, K).total;
  return CKM_OK;
}

static ckm_status check_work(const ckm_graph* g, int32_t K, void* d_work, size_t work_bytes,
                             Layout* L) {
  if (!g) return fail(CKM_E_INVALID_ARG, "graph is NULL");
  if (K < 1) return fail(CKM_E_INVALID_ARG, "K = %d < 1", K);
  if (K > CKM_MAX_CANDIDATES) return fail(CKM_E_UNSUPPORTED, "K = %d > %d", K, CKM_MAX_CANDIDATES);
  if (!d_work) return fail(CKM_E_INVALID_ARG, "work buffer is NULL");
  *L = ckm::make_layout(g->n, K);
  if (work_bytes < L->total)
    return fail(CKM_E_INVALID_ARG, "work buffer of %zu bytes, %zu needed", work_bytes, L->total);
  L->rows_on = L->rows_on && work_bytes >= L->total_rows;
  return CKM_OK;
}

ckm_status ckm_quantize_async(const ckm_graph* g, const double* d_s_frac, int64_t ld, void* d_work,
                              size_t work_bytes, void* stream) {
  Layout L;
  if (!g) return fail(CKM_E_INVALID_ARG, "graph is NULL");
  // The thresholds do not depend on K; size the check with K = 1.
  ckm_status st = check_work(g, 1, d_work, work_bytes, &L);
  if (st != CKM_OK) return st;
  if (!d_s_frac) return fail(CKM_E_INVALID_ARG, "S* is NULL");
  if (ld < g->n) return fail(CKM_E_INVALID_ARG, "ld = %lld < n = %d", (long long)ld, g->n);
  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CKM_E_DEVICE, "cannot select the graph's device %d", g->device);
  hipError_t e = ckm::launch_quantize(*g, L, d_s_frac, ld, static_cast<char*>(d_work),
                                      static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CKM_OK : fail_hip(e, "quantize launch");
}

ckm_status ckm_round_async(const ckm_graph* g, int32_t K, uint64_t seed, uint32_t flags, void* d_work,
                           size_t work_bytes, void* stream) {
  Layout L;
  ckm_status st = check_work(g, K, d_work, work_bytes, &L);
  if (st != CKM_OK) return st;
  if (flags & ~(uint32_t)CKM_F_DET0) return fail(CKM_E_INVALID_ARG, "unknown flags 0x%x", flags);
  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CKM_E_DEVICE, "cannot select the graph's device %d", g->device);
  hipError_t e = ckm::launch_round_rows(*g, L, K, seed, flags, static_cast<char*>(d_work),
                                        static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CKM_OK : fail_hip(e, "round launch");
}

static ckm_status evaluate_impl(const ckm_graph* g, int32_t K, uint64_t seed, uint32_t flags,
                                int32_t stage_splits, void* d_work, size_t work_bytes, void* stream, bool overlap) {
  Layout L;
  ckm_status st = check_work(g, K, d_work, work_bytes, &L);
  if (st != CKM_OK) return st;
  if (flags & ~(uint32_t)(CKM_F_DET0 | CKM_F_ROUNDED))
    return fail(CKM_E_INVALID_ARG, "unknown flags 0x%x", flags);
  if (stage_splits < 0) return fail(CKM_E_INVALID_ARG, "stage_splits = %d < 0", stage_splits);
  const ckm::Plan plan = stage_splits ? ckm::plan_splits(g->n, std::min(stage_splits, L.max_splits))
                                      : ckm::plan_for(g, L, K);
  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CKM_E_DEVICE, "cannot select the graph's device %d", g->device);
  hipError_t e = ckm::launch_evaluate(*g, L, K, seed, flags, plan, ckm::kSrcRound, nullptr,
                                      static_cast<char*>(d_work), static_cast<hipStream_t>(stream), overlap);
  return e == hipSuccess ? CKM_OK : fail_hip(e, "evaluate launch");
}

ckm_status ckm_evaluate_async(const ckm_graph* g, int32_t K, uint64_t seed, uint32_t flags,
                              int32_t stage_splits, void* d_work, size_t work_bytes, void* stream) {
  return evaluate_impl(g, K, seed, flags, stage_splits, d_work, work_bytes, stream, true);
}

ckm_status ckm_select_async(const ckm_graph* g, int32_t K, uint64_t seed, int64_t budget,
                            uint32_t flags, int64_t* d_peak, int64_t* d_cost, uint8_t* d_feasible,
                            int32_t* d_best_k, uint64_t* d_best_S, uint64_t* d_best_R,
                            int32_t* d_status, void* d_work, size_t work_bytes, void* stream) {
  Layout L;
  ckm_status st = check_work(g, K, d_work, work_bytes, &L);
  if (st != CKM_OK) return st;
  if (budget < 0) return fail(CKM_E_INVALID_ARG, "budget = %lld < 0", (long long)budget);
  if (flags & ~(uint32_t)(CKM_F_DET0 | CKM_F_ROUNDED))
    return fail(CKM_E_INVALID_ARG, "unknown flags 0x%x", flags);
  if (!d_peak || !d_cost || !d_feasible || !d_best_k)
    return fail(CKM_E_INVALID_ARG, "NULL peak, cost, feasible or best_k");
  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CKM_E_DEVICE, "cannot select the graph's device %d", g->device);
  hipError_t e = ckm::launch_select(*g, L, K, seed, budget, flags, d_peak, d_cost, d_feasible,
                                    d_best_k, d_best_S, d_best_R, d_status, ckm::kSrcRound, nullptr,
                                    static_cast<char*>(d_work), static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CKM_OK : fail_hip(e, "select launch");
}

ckm_status ckm_round_eval_async(const ckm_graph* g, const double* d_s_frac, int64_t ld, int32_t K,
                                uint64_t seed, int64_t budget, uint32_t flags, int64_t* d_peak,
                                int64_t* d_cost, uint8_t* d_feasible, int32_t* d_best_k,
                                uint64_t* d_best_S, uint64_t* d_best_R, int32_t* d_status,
                                void* d_work, size_t work_bytes, void* stream) {
  return ckm::round_eval(g, d_s_frac, ld, K, seed, budget, flags, d_peak, d_cost, d_feasible, d_best_k, d_best_S,
                         d_best_R, d_status, d_work, work_bytes, stream, true);
}

}  // extern "C"

ckm_status ckm::round_eval(const ckm_graph* g, const double* d_s_frac, int64_t ld, int32_t K, uint64_t seed,
                           int64_t budget, uint32_t flags, int64_t* d_peak, int64_t* d_cost, uint8_t* d_feasible,
                           int32_t* d_best_k, uint64_t* d_best_S, uint64_t* d_best_R, int32_t* d_status,
                           void* d_work, size_t work_bytes, void* stream, bool overlap) {
  Layout L;
  ckm_status st = check_work(g, K, d_work, work_bytes, &L);
  if (st != CKM_OK) return st;
  if (budget < 0) return fail(CKM_E_INVALID_ARG, "budget = %lld < 0", (long long)budget);
  if (flags & ~(uint32_t)CKM_F_DET0) return fail(CKM_E_INVALID_ARG, "unknown flags 0x%x", flags);
  if (!d_peak || !d_cost || !d_feasible || !d_best_k)
    return fail(CKM_E_INVALID_ARG, "NULL peak, cost, feasible or best_k");
  st = ckm_quantize_async(g, d_s_frac, ld, d_work, work_bytes, stream);
  if (st != CKM_OK) return st;
  st = evaluate_impl(g, K, seed, flags, 0, d_work, work_bytes, stream, overlap);
  if (st != CKM_OK) return st;
  return ckm_select_async(g, K, seed, budget, flags, d_peak, d_cost, d_feasible, d_best_k,
                          d_best_S, d_best_R, d_status, d_work, work_bytes, stream);
}

extern "C" {

ckm_status ckm_eval_schedules_async(const ckm_graph* g, const uint64_t* d_S, int32_t K, int64_t budget,
                                    int64_t* d_peak, int64_t* d_cost, uint8_t* d_feasible,
                                    int32_t* d_best_k, uint64_t* d_best_R, int32_t* d_status,
                                    void* d_work, size_t work_bytes, void* stream) {
  Layout L;
  ckm_status st = check_work(g, K, d_work, work_bytes, &L);
  if (st != CKM_OK) return st;
  if (!d_S) return fail(CKM_E_INVALID_ARG, "S is NULL");
  if (budget < 0) return fail(CKM_E_INVALID_ARG, "budget = %lld < 0", (long long)budget);
  if (!d_peak || !d_cost || !d_feasible || !d_best_k)
    return fail(CKM_E_INVALID_ARG, "NULL peak, cost, feasible or best_k");
  const ckm::Plan plan = ckm::plan_for(g, L, K);
  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CKM_E_DEVICE, "cannot select the graph's device %d", g->device);
  hipError_t e = ckm::launch_evaluate(*g, L, K, 0, 0, plan, ckm::kSrcUser, d_S, static_cast<char*>(d_work),
                                      static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail_hip(e, "evaluate launch");
  e = ckm::launch_select(*g, L, K, 0, budget, 0, d_peak, d_cost, d_feasible, d_best_k, nullptr, d_best_R,
                         d_status, ckm::kSrcUser, d_S, static_cast<char*>(d_work),
                         static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CKM_OK : fail_hip(e, "select launch");
}

ckm_status ckm_eval_schedules(const ckm_graph* g, const uint64_t* S, int32_t K, int64_t budget,
                              int64_t* peak, int64_t* cost, uint8_t* feasible, int32_t* best_k,
                              uint64_t* best_R) {
  if (!g) return fail(CKM_E_INVALID_ARG, "graph is NULL");
  if (!S || !peak || !cost || !feasible || !best_k)
    return fail(CKM_E_INVALID_ARG, "NULL S, peak, cost, feasible or best_k");
  if (K < 1) return fail(CKM_E_INVALID_ARG, "K = %d < 1", K);
  if (K > CKM_MAX_CANDIDATES) return fail(CKM_E_UNSUPPORTED, "K = %d > %d", K, CKM_MAX_CANDIDATES);
  if (budget < 0) return fail(CKM_E_INVALID_ARG, "budget = %lld < 0", (long long)budget);
  const int32_t n = g->n;
  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CKM_E_DEVICE, "cannot select the graph's device %d", g->device);
  const Layout L = ckm::make_layout(n, K);
  const int32_t W = (n + 63) / 64;
  const size_t rows_bytes = (size_t)n * W * sizeof(uint64_t);
  size_t off = 0;
  const size_t o_w = off;    off = align256(off + L.total_rows);
  const size_t o_s = off;    off = align256(off + (size_t)K * rows_bytes);
  const size_t o_peak = off; off = align256(off + (size_t)K * 8);
  const size_t o_cost = off; off = align256(off + (size_t)K * 8);
  const size_t o_feas = off; off = align256(off + (size_t)K);
  const size_t o_bk = off;   off = align256(off + 8);
  const size_t o_bR = off;   off = align256(off + rows_bytes);
  const size_t o_end = off;
  SyncCall sc(g);
  ckm_status st = sc.reserve(o_end, o_end - o_peak);
  if (st != CKM_OK) return st;
  char* d = sc.dev();
  // the matrices go straight from the caller's memory (staged by the runtime)
  const hipError_t e = hipMemcpyAsync(d + o_s, S, (size_t)K * rows_bytes, hipMemcpyHostToDevice, sc.stream());
  if (e != hipSuccess) return fail_hip(e, "hipMemcpy S");
  st = ckm_eval_schedules_async(g, reinterpret_cast<const uint64_t*>(d + o_s), K, budget,
                                reinterpret_cast<int64_t*>(d + o_peak), reinterpret_cast<int64_t*>(d + o_cost),
                                reinterpret_cast<uint8_t*>(d + o_feas), reinterpret_cast<int32_t*>(d + o_bk),
                                best_R ? reinterpret_cast<uint64_t*>(d + o_bR) : nullptr, nullptr, d + o_w, L.total_rows,
                                sc.stream());
  if (st != CKM_OK) return st;
  const Result r[] = {{peak, o_peak, (size_t)K * 8}, {cost, o_cost, (size_t)K * 8}, {feasible, o_feas, (size_t)K},
                      {best_k, o_bk, 4}, {best_R, o_bR, rows_bytes}};
  return fetch_results(sc, o_peak, o_end, 0, r, 5);
}

ckm_status ckm_threshold_eval_async(const ckm_graph* g, const double* d_s_frac, int64_t ld, const double* d_p,
                                   int32_t K, int64_t budget, int64_t* d_peak, int64_t* d_cost,
                                   uint8_t* d_feasible, int32_t* d_best_k, uint64_t* d_best_S,
                                   uint64_t* d_best_R, int32_t* d_status, void* d_work, size_t work_bytes,
                                   void* stream) {
  Layout L;
  ckm_status st = check_work(g, K, d_work, work_bytes, &L);
  if (st != CKM_OK) return st;
  if (K > CKM_MAX_THRESHOLDS) return fail(CKM_E_UNSUPPORTED, "K = %d > %d thresholds", K, CKM_MAX_THRESHOLDS);
  if (!d_s_frac || !d_p) return fail(CKM_E_INVALID_ARG, "NULL S* or thresholds");
  if (ld < g->n) return fail(CKM_E_INVALID_ARG, "ld = %lld < n = %d", (long long)ld, g->n);
  if (budget < 0) return fail(CKM_E_INVALID_ARG, "budget = %lld < 0", (long long)budget);
  if (!d_peak || !d_cost || !d_feasible || !d_best_k)
    return fail(CKM_E_INVALID_ARG, "NULL peak, cost, feasible or best_k");
  const ckm::Plan plan = ckm::plan_for(g, L, K);
  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CKM_E_DEVICE, "cannot select the graph's device %d", g->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* work = static_cast<char*>(d_work);
  hipError_t e = ckm::launch_threshold_keys(*g, L, d_s_frac, ld, d_p, K, work, s);
  if (e != hipSuccess) return fail_hip(e, "threshold key launch");
  e = ckm::launch_evaluate(*g, L, K, 0, 0, plan, ckm::kSrcThreshold, nullptr, work, s);
  if (e != hipSuccess) return fail_hip(e, "evaluate launch");
  e = ckm::launch_select(*g, L, K, 0, budget, 0, d_peak, d_cost, d_feasible, d_best_k, d_best_S, d_best_R,
                         d_status, ckm::kSrcThreshold, nullptr, work, s);
  return e == hipSuccess ? CKM_OK : fail_hip(e, "select launch");
}

ckm_status ckm_threshold_eval(const ckm_graph* g, const double* s_frac, int64_t ld, const double* p,
                              int32_t K, int64_t budget, int64_t* peak, int64_t* cost, uint8_t* feasible,
                              int32_t* best_k, uint64_t* best_S, uint64_t* best_R) {
  if (!g) return fail(CKM_E_INVALID_ARG, "graph is NULL");
  if (!s_frac || !p || !peak || !cost || !feasible || !best_k)
    return fail(CKM_E_INVALID_ARG, "NULL S*, thresholds, peak, cost, feasible or best_k");
  if (ld < g->n) return fail(CKM_E_INVALID_ARG, "ld = %lld < n = %d", (long long)ld, g->n);
  if (K < 1) return fail(CKM_E_INVALID_ARG, "K = %d < 1", K);
  if (K > CKM_MAX_THRESHOLDS) return fail(CKM_E_UNSUPPORTED, "K = %d > %d thresholds", K, CKM_MAX_THRESHOLDS);
  if (budget < 0) return fail(CKM_E_INVALID_ARG, "budget = %lld < 0", (long long)budget);
  const int32_t n = g->n;
  for (int32_t k = 0; k < K; ++k)
    if (std::isnan(p[k])) return fail(CKM_E_INVALID_ARG, "threshold %d is NaN", k);

  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CKM_E_DEVICE, "cannot select the graph's device %d", g->device);
  const Layout L = ckm::make_layout(n, K);
  const int32_t W = (n + 63) / 64;
  const size_t rows_bytes = (size_t)n * W * sizeof(uint64_t);
  const size_t s_bytes = align256((size_t)n * n * sizeof(double));
  const size_t p_bytes = align256((size_t)K * sizeof(double));
  size_t off = 0;
  const size_t o_w = off;    off = align256(off + L.total_rows);
  const size_t o_s = off;    off = align256(off + s_bytes);
  const size_t o_p = off;    off = align256(off + p_bytes);
  const size_t o_peak = off; off = align256(off + (size_t)K * 8);
  const size_t o_cost = off; off = align256(off + (size_t)K * 8);
  const size_t o_feas = off; off = align256(off + (size_t)K);
  const size_t o_bk = off;   off = align256(off + 8);
  const size_t o_bS = off;   off = align256(off + rows_bytes);
  const size_t o_bR = off;   off = align256(off + rows_bytes);
  const size_t o_end = off;
  // pinned: S*, thresholds, then the results
  SyncCall sc(g);
  ckm_status st = sc.reserve(o_end, s_bytes + p_bytes + (o_end - o_peak));
  if (st != CKM_OK) return st;
  char* d = sc.dev();
  char* h = sc.host();
  if ((st = stage_s_frac(s_frac, ld, n, reinterpret_cast<double*>(h), d + o_s, sc.stream())) != CKM_OK) return st;
  memcpy(h + s_bytes, p, (size_t)K * sizeof(double));
  const hipError_t e = hipMemcpyAsync(d + o_p, h + s_bytes, (size_t)K * sizeof(double), hipMemcpyHostToDevice,
                                      sc.stream());
  if (e != hipSuccess) return fail_hip(e, "hipMemcpy thresholds");
  st = ckm_threshold_eval_async(g, reinterpret_cast<const double*>(d + o_s), n,
                                reinterpret_cast<const double*>(d + o_p), K, budget,
                                reinterpret_cast<int64_t*>(d + o_peak), reinterpret_cast<int64_t*>(d + o_cost),
                                reinterpret_cast<uint8_t*>(d + o_feas), reinterpret_cast<int32_t*>(d + o_bk),
                                best_S ? reinterpret_cast<uint64_t*>(d + o_bS) : nullptr,
                                best_R ? reinterpret_cast<uint64_t*>(d + o_bR) : nullptr, nullptr, d + o_w, L.total_rows,
                                sc.stream());
  if (st != CKM_OK) return st;
  const Result r[] = {{peak, o_peak, (size_t)K * 8}, {cost, o_cost, (size_t)K * 8}, {feasible, o_feas, (size_t)K},
                      {best_k, o_bk, 4}, {best_S, o_bS, rows_bytes}, {best_R, o_bR, rows_bytes}};
  return fetch_results(sc, o_peak, o_end, s_bytes + p_bytes, r, 6);
}

ckm_status ckm_plan_async(const ckm_graph* g, const uint64_t* d_S, const uint64_t* d_R, uint32_t flags,
                          ckm_stmt* d_P, int64_t capacity, int64_t* d_count, int64_t* d_mem, int32_t* d_status,
                          void* d_work, size_t work_bytes, void* stream) {
  Layout L;
  ckm_status st = check_work(g, 1, d_work, work_bytes, &L);
  if (st != CKM_OK) return st;
  if (!d_S || !d_R || !d_count) return fail(CKM_E_INVALID_ARG, "NULL S, R or count");
  if (flags & ~(uint32_t)CKM_PLAN_EARLY_FREE) return fail(CKM_E_INVALID_ARG, "unknown flags 0x%x", flags);
  if (capacity < 0) return fail(CKM_E_INVALID_ARG, "capacity = %lld < 0", (long long)capacity);
  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CKM_E_DEVICE, "cannot select the graph's device %d", g->device);
  hipError_t e = ckm::launch_plan(*g, L, d_S, d_R, flags, reinterpret_cast<int32_t*>(d_P), capacity, d_count,
                                  d_P ? d_mem : nullptr, d_status, static_cast<char*>(d_work),
                                  static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CKM_OK : fail_hip(e, "plan launch");
}

ckm_status ckm_plan(const ckm_graph* g, const uint64_t* S, const uint64_t* R, uint32_t flags, ckm_stmt* P,
                    int64_t capacity, int64_t* count, int64_t* mem) {
  if (!g) return fail(CKM_E_INVALID_ARG, "graph is NULL");
  if (!S || !R || !count) return fail(CKM_E_INVALID_ARG, "NULL S, R or count");
  if (flags & ~(uint32_t)CKM_PLAN_EARLY_FREE) return fail(CKM_E_INVALID_ARG, "unknown flags 0x%x", flags);
  if (P && capacity < 0) return fail(CKM_E_INVALID_ARG, "capacity = %lld < 0", (long long)capacity);
  if (!P) capacity = 0;
  const int32_t n = g->n;
  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CKM_E_DEVICE, "cannot select the graph's device %d", g->device);
  const Layout L = ckm::make_layout(n, 1);
  const size_t rows_bytes = (size_t)n * ((n + 63) / 64) * sizeof(uint64_t);
  const size_t rows_al = align256(rows_bytes);
  size_t off = 0;
  const size_t o_w = off;   off = align256(off + L.total);
  const size_t o_s = off;   off = align256(off + rows_bytes);
  const size_t o_r = off;   off = align256(off + rows_bytes);
  const size_t o_cnt = off; off = align256(off + 8);
  const size_t o_st = off;  off = align256(off + 8);
  const size_t o_p = off;   off = align256(off + (size_t)capacity * sizeof(ckm_stmt));
  const size_t o_m = off;   off = align256(off + (mem ? (size_t)capacity * sizeof(int64_t) : 0));
  // pinned: S and R, then the count and status
  SyncCall sc(g);
  ckm_status st = sc.reserve(off, 2 * rows_al + (o_p - o_cnt));
  if (st != CKM_OK) return st;
  char* d = sc.dev();
  char* h = sc.host();
  memcpy(h, S, rows_bytes);
  memcpy(h + rows_al, R, rows_bytes);
  hipError_t e;
  if ((e = hipMemcpyAsync(d + o_s, h, rows_bytes, hipMemcpyHostToDevice, sc.stream())) != hipSuccess ||
      (e = hipMemcpyAsync(d + o_r, h + rows_al, rows_bytes, hipMemcpyHostToDevice, sc.stream())) != hipSuccess)
    return fail_hip(e, "hipMemcpy S or R");
  st = ckm_plan_async(g, reinterpret_cast<const uint64_t*>(d + o_s), reinterpret_cast<const uint64_t*>(d + o_r),
                      flags, P ? reinterpret_cast<ckm_stmt*>(d + o_p) : nullptr, capacity,
                      reinterpret_cast<int64_t*>(d + o_cnt), mem ? reinterpret_cast<int64_t*>(d + o_m) : nullptr,
                      reinterpret_cast<int32_t*>(d + o_st), d + o_w, L.total, sc.stream());
  if (st != CKM_OK) return st;
  int64_t total = 0;
  int32_t status_dev = 0;
  const Result r[] = {{&total, o_cnt, 8}, {&status_dev, o_st, 4}};
  if ((st = fetch_results(sc, o_cnt, o_p, 2 * rows_al, r, 2)) != CKM_OK) return st;
  *count = total;
  if (status_dev != CKM_OK)
    return (P && total > capacity) ? fail(CKM_E_INVALID_ARG, "plan has %lld statements, capacity %lld",
                                          (long long)total, (long long)capacity)
                                   : fail(CKM_E_INVALID_ARG, "(S, R) violates (4a), (1b), (1c) or S & R = 0");
  if (P && total > 0) {
    // the statements go straight into the caller's memory
    if ((e = hipMemcpyAsync(P, d + o_p, (size_t)total * sizeof(ckm_stmt), hipMemcpyDeviceToHost, sc.stream())) !=
            hipSuccess ||
        (mem && (e = hipMemcpyAsync(mem, d + o_m, (size_t)total * sizeof(int64_t), hipMemcpyDeviceToHost,
                                    sc.stream())) != hipSuccess))
      return fail_hip(e, "hipMemcpy plan");
    return sc.wait();
  }
  return CKM_OK;
}

ckm_status ckm_max_batch_async(const ckm_graph* g, int32_t K, int64_t budget, int64_t cost_cap, int64_t* d_batch,
                               int32_t* d_best_k, int64_t* d_best_batch, int32_t* d_status, void* d_work,
                               size_t work_bytes, void* stream) {
  Layout L;
  ckm_status st = check_work(g, K, d_work, work_bytes, &L);
  if (st != CKM_OK) return st;
  if (budget < 0) return fail(CKM_E_INVALID_ARG, "budget = %lld < 0", (long long)budget);
  if (cost_cap < 0) return fail(CKM_E_INVALID_ARG, "cost_cap = %lld < 0", (long long)cost_cap);
  if (!d_batch || !d_best_k) return fail(CKM_E_INVALID_ARG, "NULL batch or best_k");
  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CKM_E_DEVICE, "cannot select the graph's device %d", g->device);
  hipError_t e = ckm::launch_max_batch(*g, L, K, budget, cost_cap, d_batch, d_best_k, d_best_batch, d_status,
                                       static_cast<char*>(d_work), static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CKM_OK : fail_hip(e, "max batch launch");
}

ckm_status ckm_max_batch(const ckm_graph* g, const double* s_frac, int64_t ld, int32_t K, uint64_t seed,
                         uint32_t flags, int64_t budget, int64_t cost_cap, int64_t* batch, int32_t* best_k,
                         int64_t* best_batch) {
  if (!g) return fail(CKM_E_INVALID_ARG, "graph is NULL");
  if (!s_frac || !batch || !best_k) return fail(CKM_E_INVALID_ARG, "NULL S*, batch or best_k");
  if (ld < g->n) return fail(CKM_E_INVALID_ARG, "ld = %lld < n = %d", (long long)ld, g->n);
  if (K < 1) return fail(CKM_E_INVALID_ARG, "K = %d < 1", K);
  if (K > CKM_MAX_CANDIDATES) return fail(CKM_E_UNSUPPORTED, "K = %d > %d", K, CKM_MAX_CANDIDATES);
  if (budget < 0) return fail(CKM_E_INVALID_ARG, "budget = %lld < 0", (long long)budget);
  if (cost_cap < 0) return fail(CKM_E_INVALID_ARG, "cost_cap = %lld < 0", (long long)cost_cap);
  if (flags & ~(uint32_t)CKM_F_DET0) return fail(CKM_E_INVALID_ARG, "unknown flags 0x%x", flags);
  const int32_t n = g->n;
  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CKM_E_DEVICE, "cannot select the graph's device %d", g->device);
  const Layout L = ckm::make_layout(n, K);
  const size_t s_bytes = align256((size_t)n * n * sizeof(double));
  size_t off = 0;
  const size_t o_w = off;  off = align256(off + L.total_rows);
  const size_t o_s = off;  off = align256(off + s_bytes);
  const size_t o_b = off;  off = align256(off + (size_t)K * 8);
  const size_t o_bk = off; off = align256(off + 8);
  const size_t o_bb = off; off = align256(off + 8);
  const size_t o_end = off;
  SyncCall sc(g);
  ckm_status st = sc.reserve(o_end, s_bytes + (o_end - o_b));
  if (st != CKM_OK) return st;
  char* d = sc.dev();
  const hipStream_t stream = sc.stream();
  if ((st = stage_s_frac(s_frac, ld, n, reinterpret_cast<double*>(sc.host()), d + o_s, stream)) != CKM_OK ||
      (st = ckm_quantize_async(g, reinterpret_cast<const double*>(d + o_s), n, d + o_w, L.total_rows, stream)) !=
          CKM_OK ||
      (st = ckm_evaluate_async(g, K, seed, flags, 0, d + o_w, L.total_rows, stream)) != CKM_OK ||
      (st = ckm_max_batch_async(g, K, budget, cost_cap, reinterpret_cast<int64_t*>(d + o_b),
                                reinterpret_cast<int32_t*>(d + o_bk), reinterpret_cast<int64_t*>(d + o_bb), nullptr,
                                d + o_w, L.total_rows, stream)) != CKM_OK)
    return st;
  const Result r[] = {{batch, o_b, (size_t)K * 8}, {best_k, o_bk, 4}, {best_batch, o_bb, 8}};
  return fetch_results(sc, o_b, o_end, s_bytes, r, 3);
}

ckm_status ckm_round_eval(const ckm_graph* g, const double* s_frac, int64_t ld, int32_t K,
                          uint64_t seed, int64_t budget, uint32_t flags, int64_t* peak,
                          int64_t* cost, uint8_t* feasible, int32_t* best_k, uint64_t* best_S,
                          uint64_t* best_R) {
  if (!g) return fail(CKM_E_INVALID_ARG, "graph is NULL");
  if (!s_frac || !peak || !cost || !feasible || !best_k)
    return fail(CKM_E_INVALID_ARG, "NULL S*, peak, cost, feasible or best_k");
  if (ld < g->n) return fail(CKM_E_INVALID_ARG, "ld = %lld < n = %d", (long long)ld, g->n);
  if (K < 1) return fail(CKM_E_INVALID_ARG, "K = %d < 1", K);
  if (K > CKM_MAX_CANDIDATES) return fail(CKM_E_UNSUPPORTED, "K = %d > %d", K, CKM_MAX_CANDIDATES);
  if (budget < 0) return fail(CKM_E_INVALID_ARG, "budget = %lld < 0", (long long)budget);
  if (flags & ~(uint32_t)CKM_F_DET0) return fail(CKM_E_INVALID_ARG, "unknown flags 0x%x", flags);
  const int32_t n = g->n;
  DeviceGuard dg(g->device);
  if (!dg.ok) return fail(CKM_E_DEVICE, "cannot select the graph's device %d", g->device);
  const Layout L = ckm::make_layout(n, K);
  const int32_t W = (n + 63) / 64;
  const size_t s_bytes = align256((size_t)n * n * sizeof(double));
  const size_t rows_bytes = (size_t)n * W * sizeof(uint64_t);
  size_t off = 0;
  const size_t o_w = off;    off = align256(off + L.total_rows);
  const size_t o_s = off;    off = align256(off + s_bytes);
  const size_t o_peak = off; off = align256(off + (size_t)K * 8);
  const size_t o_cost = off; off = align256(off + (size_t)K * 8);
  const size_t o_feas = off; off = align256(off + (size_t)K);
  const size_t o_bk = off;   off = align256(off + 8);
  const size_t o_st = off;   off = align256(off + 8);
  const size_t o_bS = off;   off = align256(off + rows_bytes);
  const size_t o_bR = off;   off = align256(off + rows_bytes);
  const size_t o_end = off;
  // pinned: S*, then the results
  SyncCall sc(g);
  ckm_status st = sc.reserve(o_end, s_bytes + (o_end - o_peak));
  if (st != CKM_OK) return st;
  char* d = sc.dev();
  if ((st = stage_s_frac(s_frac, ld, n, reinterpret_cast<double*>(sc.host()), d + o_s, sc.stream())) != CKM_OK)
    return st;
  st = ckm_round_eval_async(g, reinterpret_cast<const double*>(d + o_s), n, K, seed, budget, flags,
                            reinterpret_cast<int64_t*>(d + o_peak), reinterpret_cast<int64_t*>(d + o_cost),
                            reinterpret_cast<uint8_t*>(d + o_feas), reinterpret_cast<int32_t*>(d + o_bk),
                            best_S ? reinterpret_cast<uint64_t*>(d + o_bS) : nullptr,
                            best_R ? reinterpret_cast<uint64_t*>(d + o_bR) : nullptr,
                            reinterpret_cast<int32_t*>(d + o_st), d + o_w, L.total_rows, sc.stream());
  if (st != CKM_OK) return st;
  int32_t status_dev = 0;
  const Result r[] = {{peak, o_peak, (size_t)K * 8}, {cost, o_cost, (size_t)K * 8}, {feasible, o_feas, (size_t)K},
                      {best_k, o_bk, 4}, {&status_dev, o_st, 4}, {best_S, o_bS, rows_bytes},
                      {best_R, o_bR, rows_bytes}};
  if ((st = fetch_results(sc, o_peak, o_end, s_bytes, r, 7)) != CKM_OK) return st;
  return status_dev == CKM_OK ? CKM_OK : fail((ckm_status)status_dev, "S* holds a NaN");
}

}  // extern "C"
