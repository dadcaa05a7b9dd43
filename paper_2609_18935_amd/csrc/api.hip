// Host side of the tail-update library: argument and range verification, launch
// planning, workspace carving and the C ABI declared in include/tailupdate.h.
//
// Every check runs before the first launch, so an error leaves device buffers and
// host metadata untouched (Section 4.2 of the paper: deletion ranges are verified
// against the live spans before anything is removed).
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"
#include "tailupdate.h"

namespace tu {
namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return TU_OK;
}

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

// Carves aligned regions out of a workspace; with base == nullptr it only measures.
struct Arena {
  char* base;
  size_t used = 0;
  explicit Arena(void* b) : base(static_cast<char*>(b)) {}
  void* take(size_t bytes) {
    void* p = base ? base + used : nullptr;
    used += align_up(bytes);
    return p;
  }
};

// The first kStatusBytes of every workspace hold the call's status: the tagged 64-bit
// word and, 64 bytes further, the number of the call that last ran there (CallStatus in
// common.h); the rest is carved by the planners.
constexpr size_t kStatusBytes = 256;
constexpr size_t kStatusLastOffset = 64;
std::atomic<uint32_t> g_calls{0};

// The status of a new call on workspace ws: numbers 1 .. 2^32 - 2, one per call of the process.
CallStatus call_status(void* ws) {
  uint32_t n;
  do n = g_calls.fetch_add(1, std::memory_order_relaxed) + 1;
  while (n == 0 || n == 0xFFFFFFFFu);
  CallStatus st{};
  st.word = static_cast<unsigned long long*>(ws);
  st.last = reinterpret_cast<uint32_t*>(static_cast<char*>(ws) + kStatusLastOffset);
  st.call = n;
  return st;
}
inline void* after_status(void* ws) { return ws ? static_cast<char*>(ws) + kStatusBytes : nullptr; }

// ------------------------------------------------------------------ metadata checks

int check_seq(const tu_seq* s) {
  if (!s) return fail(TU_ERR_ARG, "null context");
  if (s->len < 0 || s->capacity < s->len) return fail(TU_ERR_ARG, "len %lld outside [0, capacity %lld]",
                                                      (long long)s->len, (long long)s->capacity);
  if (s->n_live < 0 || s->n_live > s->live_cap) return fail(TU_ERR_ARG, "n_live outside [0, live_cap]");
  if (s->n_live > 0 && !s->live) return fail(TU_ERR_ARG, "null live-interval array");
  if (s->capacity > 0 && !s->d_pos) return fail(TU_ERR_ARG, "null d_pos");
  if (s->next_pos < 0 || s->next_pos > INT32_MAX) return fail(TU_ERR_ARG, "cursor outside the int32 position range");
  if (s->vt_rows < 0) return fail(TU_ERR_ARG, "negative vt_rows");
  int64_t total = 0, max_end = -1;
  for (int i = 0; i < s->n_live; ++i) {
    const tu_interval& iv = s->live[i];
    if (iv.end <= iv.begin || iv.begin < 0) return fail(TU_ERR_ARG, "empty or negative live run");
    if (i > 0 && iv.begin == s->live[i - 1].end)
      return fail(TU_ERR_ARG, "consecutive live runs %d and %d are position-contiguous (not merged)", i - 1, i);
    max_end = std::max(max_end, iv.end);
    total += iv.end - iv.begin;
  }
  if (max_end > s->next_pos) return fail(TU_ERR_ARG, "live position at or beyond the cursor");
  if (total != s->len) return fail(TU_ERR_ARG, "live runs cover %lld positions, len is %lld",
                                   (long long)total, (long long)s->len);
  std::vector<tu_interval> sorted(s->live, s->live + s->n_live);
  std::sort(sorted.begin(), sorted.end(), [](const tu_interval& x, const tu_interval& y) { return x.begin < y.begin; });
  for (size_t i = 1; i < sorted.size(); ++i)
    if (sorted[i].begin < sorted[i - 1].end) return fail(TU_ERR_ARG, "live runs overlap");
  return TU_OK;
}

// The live runs sorted by position, each with the cache row of its first position.
struct RunIndex {
  std::vector<tu_interval> run;   // sorted by begin
  std::vector<int64_t> row;       // first row of run[i]
  explicit RunIndex(const tu_interval* live, int n) {
    std::vector<int64_t> row0(n + 1, 0);
    for (int i = 0; i < n; ++i) row0[i + 1] = row0[i] + (live[i].end - live[i].begin);
    std::vector<int> order(n);
    for (int i = 0; i < n; ++i) order[i] = i;
    std::sort(order.begin(), order.end(), [&](int x, int y) { return live[x].begin < live[y].begin; });
    for (int i : order) {
      run.push_back(live[i]);
      row.push_back(row0[i]);
    }
  }
  // index of the run holding position p, or -1
  int find(int64_t p) const {
    int lo = 0, hi = (int)run.size() - 1;
    while (lo <= hi) {
      const int mid = (lo + hi) / 2;
      if (run[mid].end <= p) lo = mid + 1;
      else if (run[mid].begin > p) hi = mid - 1;
      else return mid;
    }
    return -1;
  }
};

// Appends a run in row order, merging it into the previous run when contiguous.
void push_run(std::vector<tu_interval>& iv, int64_t begin, int64_t end) {
  if (end <= begin) return;
  if (!iv.empty() && iv.back().end == begin) iv.back().end = end;
  else iv.push_back({begin, end});
}

// Result of range verification for one context.
struct RangeCheck {
  int64_t removed = 0;
  int64_t first_row = 0;                  // first removed cache row
  // removed rows as (first row, length) spans, sorted by row; a range whose positions
  // sit in several runs maps to several spans
  std::vector<std::pair<int64_t, int64_t>> spans;
  std::vector<tu_interval> live_after;    // runs after the removal, in row order
};

// Positions [a, b) as cache-row spans, appended to `spans`; false if a position is not live.
bool range_rows(const RunIndex& ri, int64_t a, int64_t b, std::vector<std::pair<int64_t, int64_t>>* spans) {
  int at = ri.find(a);
  while (a < b) {
    if (at < 0 || at >= (int)ri.run.size() || ri.run[at].begin > a) return false;
    const int64_t e = std::min(b, ri.run[at].end);
    spans->push_back({ri.row[at] + (a - ri.run[at].begin), e - a});
    a = e;
    ++at;   // the next run by position must start where this one ends
  }
  return true;
}

// The runs of `live` (row order) minus position ranges (sorted, disjoint), in row order.
std::vector<tu_interval> subtract_runs(const tu_interval* live, int n_live, const int64_t* ranges, int n) {
  std::vector<tu_interval> out;
  for (int i = 0; i < n_live; ++i) {
    int64_t cur = live[i].begin;
    const int64_t end = live[i].end;
    // first range ending after this run's start
    int lo = 0, hi = n;
    while (lo < hi) {
      const int mid = (lo + hi) / 2;
      if (ranges[2 * mid + 1] <= cur) lo = mid + 1;
      else hi = mid;
    }
    for (int q = lo; q < n && ranges[2 * q] < end; ++q) {
      push_run(out, cur, std::max(cur, ranges[2 * q]));
      cur = std::max(cur, ranges[2 * q + 1]);
    }
    push_run(out, cur, end);
  }
  return out;
}

int check_ranges(const tu_seq* s, const int64_t* ranges, int n, RangeCheck* out) {
  if (n < 0) return fail(TU_ERR_ARG, "negative range count");
  if (n > 0 && !ranges) return fail(TU_ERR_ARG, "null ranges");
  if (n > TU_MAX_RANGES) return fail(TU_ERR_ARG, "more than %d ranges in one call", TU_MAX_RANGES);
  out->removed = 0;
  out->first_row = s->len;
  out->spans.clear();
  int64_t prev_end = INT64_MIN;
  const RunIndex ri(s->live, s->n_live);
  for (int q = 0; q < n; ++q) {
    const int64_t a = ranges[2 * q], b = ranges[2 * q + 1];
    if (b <= a) return fail(TU_ERR_RANGE, "range %d [%lld,%lld) is empty", q, (long long)a, (long long)b);
    if (a < prev_end) return fail(TU_ERR_RANGE, "ranges are not sorted and disjoint (range %d)", q);
    if (a < 0 || b > s->next_pos)
      return fail(TU_ERR_RANGE, "range %d [%lld,%lld) reaches past the cursor %lld", q, (long long)a,
                  (long long)b, (long long)s->next_pos);
    if (!range_rows(ri, a, b, &out->spans))
      return fail(TU_ERR_RANGE, "range %d [%lld,%lld) is not live", q, (long long)a, (long long)b);
    out->removed += b - a;
    prev_end = b;
  }
  if ((int)out->spans.size() > TU_MAX_RANGES)
    return fail(TU_ERR_RANGE, "the ranges map to %d row spans, more than %d", (int)out->spans.size(), TU_MAX_RANGES);
  std::sort(out->spans.begin(), out->spans.end());
  // merge row-adjacent spans (positions of two runs removed back to back)
  std::vector<std::pair<int64_t, int64_t>> merged;
  for (auto& sp : out->spans) {
    if (!merged.empty() && merged.back().first + merged.back().second == sp.first) merged.back().second += sp.second;
    else merged.push_back(sp);
  }
  out->spans.swap(merged);
  if (!out->spans.empty()) out->first_row = out->spans[0].first;
  out->live_after = subtract_runs(s->live, s->n_live, ranges, n);
  return TU_OK;
}

// Position runs (host [n][2]) that a placement gives the T tail tokens: non-empty,
// disjoint, free of `live` positions, below 2^31 - 1, lengths summing to T.
int check_place_runs(const int64_t* runs, int n, int64_t T, const std::vector<tu_interval>& live, int s) {
  if (n < 0 || n > TU_MAX_PLACE_RUNS) return fail(TU_ERR_ARG, "context %d: 0 .. %d placement runs", s, TU_MAX_PLACE_RUNS);
  if (n > 0 && !runs) return fail(TU_ERR_ARG, "context %d: null placement runs", s);
  int64_t total = 0;
  std::vector<tu_interval> all(live);
  for (int q = 0; q < n; ++q) {
    const int64_t a = runs[2 * q], b = runs[2 * q + 1];
    if (b <= a || a < 0 || b > INT32_MAX)
      return fail(TU_ERR_RANGE, "context %d: placement run %d [%lld,%lld) empty or outside [0, 2^31 - 1)", s, q,
                  (long long)a, (long long)b);
    total += b - a;
    all.push_back({a, b});
  }
  if (total != T) return fail(TU_ERR_ARG, "context %d: placement runs hold %lld positions, T is %lld", s,
                              (long long)total, (long long)T);
  std::sort(all.begin(), all.end(), [](const tu_interval& x, const tu_interval& y) { return x.begin < y.begin; });
  for (size_t i = 1; i < all.size(); ++i)
    if (all[i].begin < all[i - 1].end)
      return fail(TU_ERR_RANGE, "context %d: placement positions overlap each other or live positions", s);
  return TU_OK;
}

int check_attn(const tu_attn_params* p) {
  if (!p) return fail(TU_ERR_ARG, "null attention parameters");
  if (p->n_kv_heads <= 0 || p->n_q_heads <= 0 || p->n_q_heads % p->n_kv_heads)
    return fail(TU_ERR_ARG, "n_q_heads must be a positive multiple of n_kv_heads");
  if (p->head_dim != 64 && p->head_dim != 128 && p->head_dim != 256)
    return fail(TU_ERR_ARG, "head_dim must be 64, 128 or 256");
  if (p->rotary_dim < 0 || p->rotary_dim > p->head_dim || (p->rotary_dim & 1))
    return fail(TU_ERR_ARG, "rotary_dim must be even and within [0, head_dim]");
  if (!(p->rope_theta > 0.0) || !std::isfinite(p->rope_theta)) return fail(TU_ERR_ARG, "rope_theta must be positive");
  if (!(p->softmax_scale > 0.f) || !std::isfinite(p->softmax_scale)) return fail(TU_ERR_ARG, "softmax_scale must be positive");
  if (p->kv_splits < 0 || p->kv_splits > 64) return fail(TU_ERR_ARG, "kv_splits must be in [0, 64]");
  if ((long)p->n_kv_heads * p->head_dim * 2 > kGatherStripeBytes) return fail(TU_ERR_ARG, "cache row too wide");
  return TU_OK;
}

int check_delta(const tu_delta_params* p) {
  if (!p) return fail(TU_ERR_ARG, "null delta parameters");
  if (p->n_k_heads <= 0 || p->n_v_heads <= 0 || p->n_v_heads % p->n_k_heads)
    return fail(TU_ERR_ARG, "n_v_heads must be a positive multiple of n_k_heads");
  if (p->d_k != p->d_v || (p->d_k != 64 && p->d_k != 128)) return fail(TU_ERR_ARG, "d_k = d_v must be 64 or 128");
  if (p->chunk != 16 && p->chunk != 32 && p->chunk != 64) return fail(TU_ERR_ARG, "chunk must be 16, 32 or 64");
  if (!std::isfinite(p->scale)) return fail(TU_ERR_ARG, "scale must be finite");
  return TU_OK;
}

int hip_check(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(TU_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return TU_OK;
}

// ------------------------------------------------------------------ kernel timing

struct ProfRec {
  const char* name;
  hipEvent_t start;
  hipEvent_t stop;
};
thread_local bool g_prof = false;
thread_local std::vector<ProfRec> g_recs;
thread_local uint64_t g_launches = 0;   // kernels this thread has enqueued through timed()

// Runs `launch` (which enqueues one kernel on `st`), bracketed by events when profiling.
template <class F>
hipError_t timed(const char* name, hipStream_t st, F&& launch) {
  ++g_launches;
  if (!g_prof) return launch();
  ProfRec r{name, nullptr, nullptr};
  if (hipEventCreate(&r.start) != hipSuccess) return launch();
  if (hipEventCreate(&r.stop) != hipSuccess) {
    (void)hipEventDestroy(r.start);
    return launch();
  }
  (void)hipEventRecord(r.start, st);
  const hipError_t e = launch();
  (void)hipEventRecord(r.stop, st);
  g_recs.push_back(r);
  return e;
}

// ------------------------------------------------------------------ compaction plan

struct CompactItem {
  tu_seq* seq;
  const int64_t* ranges;
  int n_ranges;
  RangeCheck rc;
  int32_t* src_index;        // device, caller's or workspace
  bool user_index = false;   // the caller asked for src_index
  bool scan = true;          // run the keep-scan (src_index, position check)
  std::vector<void*> bufs;   // K and V of every attention layer
};

struct CompactPlan {
  std::vector<CompactArgs> launches;
  size_t ws_bytes = 0;
};

// Builds the compaction launches for a set of contexts. With ws == nullptr only the
// workspace size is computed.
int plan_compaction(std::vector<CompactItem>& items, int row_bytes, void* ws, const CallStatus& status,
                    CompactPlan* plan) {
  Arena ar(ws);
  const int R = kGatherStripeBytes / row_bytes;
  const int64_t align_rows = std::max(1, 128 / row_bytes);
  for (auto& it : items) {   // src_index storage
    void* p = ar.take(sizeof(int32_t) * std::max<int64_t>(1, it.seq->len));
    it.user_index = it.src_index != nullptr && it.src_index != p;
    if (!it.user_index) it.src_index = static_cast<int32_t*>(p);
  }
  // launch groups of (context, buffer range, scan?, move?) entries
  struct Entry {
    int item, buf0, nbuf;
    bool scan, move;
  };
  std::vector<std::vector<Entry>> groups;
  {
    std::vector<Entry> cur;
    int bufs = 0, nr = 0, ns = 0;
    auto flush = [&] {
      if (!cur.empty()) groups.push_back(cur);
      cur.clear();
      bufs = nr = ns = 0;
    };
    for (int i = 0; i < (int)items.size(); ++i) {
      const auto& it = items[i];
      const bool moves = it.rc.removed > 0 && it.seq->len - it.rc.removed > it.rc.first_row && !it.bufs.empty();
      const bool scans = it.scan && it.seq->len > 0 && (it.rc.removed > 0 || it.user_index);
      if (!moves && !scans) continue;
      int b0 = 0;
      bool first = true;
      do {
        const int nb = moves ? std::min<int>(kMaxBufPerLaunch, (int)it.bufs.size() - b0) : 0;
        const bool sc = scans && first;
        if ((int)cur.size() == kMaxSeqPerCompact || bufs + nb > kMaxBufPerLaunch ||
            (sc && nr + it.n_ranges > kMaxRangesPerLaunch) || (ns + (int)it.rc.spans.size() > kMaxRangesPerLaunch))
          flush();
        cur.push_back({i, b0, nb, sc, moves});
        bufs += nb;
        if (sc) nr += it.n_ranges;
        ns += (int)it.rc.spans.size();   // spans are referenced by both the scan and the move entries
        b0 += nb;
        first = false;
      } while (moves && b0 < (int)it.bufs.size());
    }
    flush();
  }
  plan->launches.clear();
  const int max_blocks = ws ? compact_max_blocks() : 0;
  for (auto& g : groups) {
    CompactArgs a{};
    a.rows_per_stripe = R;
    a.row_bytes = row_bytes;
    int nr = 0, ns = 0, items_total = 0, flag_off = 0, nbufs = 0;
    std::vector<int> span_at(items.size(), -1);   // where each context's spans sit in this launch
    auto spans_of = [&](const CompactItem& it, int idx) {
      if (span_at[idx] >= 0) return span_at[idx];
      span_at[idx] = ns;
      int64_t before = 0;
      const int n_sp = (int)it.rc.spans.size();
      for (int q = 0; q < n_sp; ++q) {
        a.spans[ns + q][0] = (int32_t)(it.rc.spans[q].first - before);
        a.spans[ns + q][1] = (int32_t)it.rc.spans[q].second;
        before += it.rc.spans[q].second;
      }
      ns += n_sp;
      return span_at[idx];
    };
    for (auto& e : g) {
      const auto& it = items[e.item];
      if (e.scan) {
        ScanSeq& c = a.scan[a.n_scan++];
        c.pos = it.seq->d_pos;
        c.src_index = it.src_index;
        c.L_old = (int32_t)it.seq->len;
        c.range_begin = nr;
        c.n_ranges = it.n_ranges;
        c.span_begin = spans_of(it, e.item);
        c.n_spans = (int32_t)it.rc.spans.size();
        c.block_begin = a.n_scan_blocks;
        a.n_scan_blocks += (int32_t)((it.seq->len + kScanRows - 1) / kScanRows);
        for (int q = 0; q < it.n_ranges; ++q) {
          a.ranges[nr + q][0] = (int32_t)it.ranges[2 * q];
          a.ranges[nr + q][1] = (int32_t)it.ranges[2 * q + 1];
        }
        nr += it.n_ranges;
      }
      if (e.move && e.nbuf > 0) {
        GatherSeq& m = a.seq[a.n_seq++];
        const int64_t n_keep = it.seq->len - it.rc.removed;
        const int64_t rb = (it.rc.first_row / align_rows) * align_rows;
        const bool with_pos = e.buf0 == 0;   // the context's first buffer group also moves positions
        m.pos = with_pos ? it.seq->d_pos : nullptr;
        m.row_begin = (int32_t)rb;
        m.n_keep = (int32_t)n_keep;
        m.n_stripes = (int32_t)((n_keep - rb + R - 1) / R);
        m.item_begin = items_total;
        m.buf_begin = nbufs;
        m.n_buf = e.nbuf;
        m.flag_begin = flag_off;
        m.window = (int32_t)((it.rc.removed + R - 1 + R - 1) / R);
        m.span_begin = spans_of(it, e.item);
        m.n_spans = (int32_t)it.rc.spans.size();
        for (int b = 0; b < e.nbuf; ++b) a.bufs[nbufs++] = it.bufs[e.buf0 + b];
        items_total += m.n_stripes * m.n_buf;
        flag_off += m.n_stripes;
      }
    }
    a.total_items = items_total;
    a.n_flag_words = flag_off * kFlagStride;
    // gather workgroups claim items in order, so any count works; one grid's worth of
    // resident workgroups suffices (the sizing pass, without a device, takes the cap)
    a.n_workers = std::min({items_total, kMaxGatherWorkers, ws ? std::max(1, max_blocks) : kMaxGatherWorkers});
    // [claim counter | stripe counters], one 128-byte line apart
    a.n_counter_words = kFlagStride + a.n_flag_words;
    int32_t* words = static_cast<int32_t*>(ar.take(sizeof(int32_t) * (size_t)a.n_counter_words));
    a.claim = words;
    a.flags = words ? words + kFlagStride : nullptr;
    a.status = status;
    plan->launches.push_back(a);
  }
  plan->ws_bytes = ar.used;
  if (ws && max_blocks <= 8) return fail(TU_ERR_HIP, "cannot size the compaction grid");
  return TU_OK;
}

int run_compaction(const CompactPlan& plan, hipStream_t st) {
  for (size_t i = 0; i < plan.launches.size(); ++i)
    if (int e = hip_check(timed("compact", st, [&] { return launch_compact(plan.launches[i], st); }),
                          "compaction launch"))
      return e;
  return TU_OK;
}

// ------------------------------------------------------------------ attention plan

struct AttnItem {
  const tu_seq* seq;
  int64_t L_keep;           // surviving rows (new rows are appended at L_keep)
  int64_t T;
  int64_t cursor;
  void* k_cache;
  void* v_cache;
  const bf16_t* q;
  const bf16_t* k;
  const bf16_t* v;
  float* out;
  bf16_t* q_hat;            // caller's or null (workspace)
  const int64_t* place_runs = nullptr;   // slot placement: host [n][2] position runs of the tail
  int n_place_runs = 0;
  void* vt_cache = nullptr;  // persistent V^T copy of the layer, or null (packed into the workspace)
  int64_t vt_rows = 0;       // rows of the copy that are current (before this call's append)
};

struct AttnLaunch {
  RopeArgs rope;
  int rope_tokens;
  PackArgs pack;
  AttnArgs attn;
  AttnOrder order;
  MergeArgs merge;
  int merge_rows;
};

inline int64_t vt_head_tiles(int64_t rows) { return (rows + kAttnKeys - 1) / kAttnKeys; }

// Key-range splits of one context's attention. An attention workgroup holds a whole CU,
// so a launch runs in waves of kCus workgroups. When every item of the launch has the
// same surviving rows and tail (one context, or the attention layers of one context's
// stack), the split count minimises (waves) x (time of one workgroup: its key tiles plus
// a fixed part) plus the merge (a launch, and the partial outputs written and read back
// once per split); about 3.8 us per 64-key tile of 256 rows at head_dim 256, 5 TB/s. With items of
// different lengths in the launch (whose waves do not line up) it takes enough splits
// for the launch to fill the CUs. At least 4 key tiles per split, at most
// kMaxAutoSplits (a decode-like tail of one token over 32K rows fills the chip with 128
// splits of its two KV heads).
constexpr int kMaxAutoSplits = 128;
constexpr int kGateWaves = 4;   // attention launches this many CU-waves long wait for the delta layers

int choose_splits(const tu_attn_params* p, int64_t L_keep, int64_t T, int64_t base_items_total, bool uniform) {
  if (p->kv_splits > 0) return p->kv_splits;
  const int64_t n_kt = (L_keep + T + kAttnKeys - 1) / kAttnKeys;
  const int64_t max_s = std::max<int64_t>(1, std::min<int64_t>(kMaxAutoSplits, n_kt / 4));
  if (!uniform) {
    const int64_t want = std::max<int64_t>(1, (kCus + base_items_total - 1) / std::max<int64_t>(1, base_items_total));
    return (int)std::min(want, max_s);
  }
  const double tile_us = 3.8 * p->head_dim / 256.0;
  const double split_us = (double)T * p->n_q_heads * p->head_dim * 4.0 / 5e6;
  double best = 0.0;
  int best_s = 1;
  for (int64_t s = 1; s <= max_s; ++s) {
    const int64_t waves = (base_items_total * s + kCus - 1) / kCus;
    const double est = (double)waves * ((double)((n_kt + s - 1) / s) * tile_us + 5.0) + (s > 1 ? 5.0 + split_us * s : 0.0);
    if (s == 1 || est < best) {
      best = est;
      best_s = (int)s;
    }
  }
  return best_s;
}

// Die table of a launch of several contexts: groups (context, kv head, split) cost their
// items' key tiles plus one each; longest first, each goes to the die with the least
// cost so far, and each die runs its groups in that order. Launches of one context, and
// launches with more groups than the table holds, keep the equal-share remap.
void plan_dies(const AttnArgs& a, int G, AttnOrder* o) {
  o->n_groups = 0;
  o->blocks = 0;
  if (a.n_seq < 2) return;
  struct Grp {
    int64_t cost;
    int32_t item0, count;
  };
  std::vector<Grp> gs;
  for (int si = 0; si < a.n_seq; ++si) {
    const AttnSeq& s = a.seq[si];
    for (int sp = 0; sp < s.n_splits; ++sp) {
      int64_t cost = 0;
      for (int q = 0; q < s.n_tiles; ++q) {
        const int64_t r_last = std::min<int64_t>((int64_t)s.T * G, (int64_t)(q + 1) * kAttnRows) - 1;
        const int64_t n_kt = (s.L_keep + r_last / G + 1 + kAttnKeys - 1) / kAttnKeys;
        const int64_t tps = (n_kt + s.n_splits - 1) / s.n_splits;
        cost += std::max<int64_t>(0, std::min(n_kt, sp * tps + tps) - sp * tps) + 1;
      }
      for (int h = 0; h < a.n_kv_heads; ++h)
        gs.push_back({cost, s.item_begin + (h * s.n_splits + sp) * s.n_tiles, s.n_tiles});
    }
  }
  if ((int)gs.size() > kMaxAttnGroups || a.total_items > 65535) return;
  std::stable_sort(gs.begin(), gs.end(), [](const Grp& x, const Grp& y) { return x.cost > y.cost; });
  int64_t load[kXcds] = {};
  std::vector<int> die(gs.size());
  for (size_t g = 0; g < gs.size(); ++g) {
    int x = 0;
    for (int y = 1; y < kXcds; ++y)
      if (load[y] < load[x]) x = y;
    die[g] = x;
    load[x] += gs[g].cost;
  }
  int n = 0, most = 0;
  for (int x = 0; x < kXcds; ++x) {
    o->die_begin[x] = n;
    int slots = 0;
    for (size_t g = 0; g < gs.size(); ++g)
      if (die[g] == x) {
        o->grp_item0[n] = (uint16_t)gs[g].item0;
        slots += gs[g].count;
        o->grp_end[n++] = (uint16_t)std::min(slots, 65535);
      }
    most = std::max(most, slots);
  }
  if (most > 65535) {   // slot counts are 16-bit: keep the equal-share order
    o->n_groups = 0;
    o->blocks = 0;
    return;
  }
  o->die_begin[kXcds] = n;
  o->n_groups = n;
  o->blocks = most * kXcds;
}

int plan_attention(const tu_attn_params* p, std::vector<AttnItem>& items, void* ws, const CallStatus& status,
                   std::vector<AttnLaunch>* out, size_t* ws_bytes) {
  const int Hq = p->n_q_heads, Hkv = p->n_kv_heads, D = p->head_dim, G = Hq / Hkv;
  size_t max_used = 0;
  out->clear();
  for (size_t g0 = 0, g1 = 0; g0 < items.size(); g0 = g1) {
    // up to kMaxSeqPerLaunch contexts and kMaxPlaceRunsPerLaunch placement runs per launch
    int runs = 0;
    while (g1 < items.size() && g1 - g0 < (size_t)kMaxSeqPerLaunch &&
           runs + items[g1].n_place_runs <= kMaxPlaceRunsPerLaunch)
      runs += items[g1++].n_place_runs;
    Arena ar(ws);
    int64_t base_items = 0;
    bool uniform = true;   // every item with a tail has the same surviving rows and tail length
    const AttnItem* first = nullptr;
    for (size_t i = g0; i < g1; ++i) {
      base_items += (int64_t)Hkv * ((items[i].T * G + kAttnRows - 1) / kAttnRows);
      if (items[i].T <= 0) continue;
      if (!first) first = &items[i];
      uniform = uniform && items[i].T == first->T && items[i].L_keep == first->L_keep;
    }
    AttnLaunch L{};
    L.rope.n_q_heads = Hq;
    L.rope.n_kv_heads = Hkv;
    L.rope.head_dim = D;
    L.rope.rotary_dim = p->rotary_dim;
    L.rope.theta = p->rope_theta;
    L.attn.n_q_heads = Hq;
    L.attn.n_kv_heads = Hkv;
    L.attn.scale_log2 = p->softmax_scale * 1.4426950408889634f;
    L.merge.n_q_heads = Hq;
    int tok = 0, item_total = 0, pack_total = 0, mrows = 0, n_runs = 0;
    for (size_t i = g0; i < g1; ++i) {
      const AttnItem& it = items[i];
      if (it.T <= 0) continue;
      bf16_t* qh = it.q_hat;
      void* qh_ws = ar.take(sizeof(bf16_t) * it.T * Hq * D);
      if (!qh) qh = static_cast<bf16_t*>(qh_ws);
      const int tiles = (int)((it.T * G + kAttnRows - 1) / kAttnRows);
      const int splits = choose_splits(p, it.L_keep, it.T, base_items, uniform);
      // V^T tiles: refreshed in the layer's own copy from the first row it lacks, or all
      // packed into the workspace
      const int vt_end = (int)vt_head_tiles(it.L_keep + it.T);
      _Float16* vt;
      int vt_begin, head_tiles;
      if (it.vt_cache) {
        vt = static_cast<_Float16*>(it.vt_cache);
        head_tiles = (int)vt_head_tiles(it.seq->capacity);
        vt_begin = (int)(std::min(it.vt_rows, it.L_keep) / kAttnKeys);
      } else {
        vt = static_cast<_Float16*>(ar.take(sizeof(_Float16) * (size_t)Hkv * vt_end * D * kVtRow));
        head_tiles = vt_end;
        vt_begin = 0;
      }
      _Float16* po = nullptr;
      float* pml = nullptr;
      if (splits > 1) {
        po = static_cast<_Float16*>(ar.take(sizeof(_Float16) * splits * it.T * Hq * D));
        pml = static_cast<float*>(ar.take(sizeof(float) * 2 * splits * it.T * Hq));
      }
      RopeSeq& r = L.rope.seq[L.rope.n_seq++];
      r.q = it.q;
      r.k = it.k;
      r.v = it.v;
      r.q_hat = qh;
      r.k_cache = static_cast<bf16_t*>(it.k_cache);
      r.v_cache = static_cast<bf16_t*>(it.v_cache);
      r.pos = it.seq->d_pos;
      r.cursor = it.cursor;
      r.L_keep = (int32_t)it.L_keep;
      r.T = (int32_t)it.T;
      r.tok_begin = tok;
      r.run_begin = n_runs;
      r.n_runs = it.n_place_runs;
      for (int q = 0, t0 = 0; q < it.n_place_runs; ++q) {
        L.rope.runs[n_runs][0] = (int32_t)it.place_runs[2 * q];
        L.rope.runs[n_runs][1] = t0;
        t0 += (int)(it.place_runs[2 * q + 1] - it.place_runs[2 * q]);
        ++n_runs;
      }
      tok += (int)it.T;
      PackSeq& pk = L.pack.seq[L.pack.n_seq++];
      pk.vt = vt;
      pk.tile_begin = vt_begin;
      pk.tile_end = vt_end;
      pk.head_tiles = head_tiles;
      pk.pack_begin = pack_total;
      pack_total += Hkv * (vt_end - vt_begin);
      AttnSeq& s = L.attn.seq[L.attn.n_seq++];
      s.q_hat = qh;
      s.k_cache = static_cast<const bf16_t*>(it.k_cache);
      s.vt = vt;
      s.out = it.out;
      s.part_o = po;
      s.part_ml = pml;
      s.L_keep = (int32_t)it.L_keep;
      s.T = (int32_t)it.T;
      s.n_tiles = tiles;
      s.n_splits = splits;
      s.item_begin = item_total;
      s.head_tiles = head_tiles;
      item_total += Hkv * splits * tiles;
      if (splits > 1) {
        L.merge.row_begin[L.merge.n_seq] = mrows;
        L.merge.seq[L.merge.n_seq++] = s;
        mrows += (int)(it.T * Hq);
      }
    }
    L.merge.row_begin[L.merge.n_seq] = mrows;
    L.rope_tokens = tok;
    L.attn.total_items = item_total;
    plan_dies(L.attn, G, &L.order);
    L.pack.pack_items = pack_total;
    L.pack.status = status;
    L.merge_rows = mrows;
    {   // lanes per row piece: one per batch of 8 splits of the launch's largest split count
      int most = 1;
      for (int m = 0; m < L.merge.n_seq; ++m) most = std::max(most, (int)L.merge.seq[m].n_splits);
      L.merge.split_lanes = most <= 8 ? 1 : most <= 16 ? 2 : most <= 32 ? 4 : 8;
    }
    max_used = std::max(max_used, ar.used);
    if (L.rope.n_seq > 0) out->push_back(L);
  }
  *ws_bytes = max_used;
  return TU_OK;
}

// Side stream of the current device for the calling thread (created on first use,
// default priority, kept for the life of the thread) with the two events that fork
// work onto it and join it back.
struct SideStream {
  hipStream_t stream = nullptr;
  hipEvent_t fork = nullptr;
  hipEvent_t join = nullptr;
};

int side_stream(SideStream** out) {
  thread_local SideStream per_device[64];
  int dev = 0;
  if (int e = hip_check(hipGetDevice(&dev), "current device")) return e;
  if (dev < 0 || dev >= 64) return fail(TU_ERR_HIP, "device index %d out of range", dev);
  SideStream& s = per_device[dev];
  if (!s.stream) {
    if (int e = hip_check(hipStreamCreateWithFlags(&s.stream, hipStreamNonBlocking), "side stream")) return e;
    if (int e = hip_check(hipEventCreateWithFlags(&s.fork, hipEventDisableTiming), "fork event")) return e;
    if (int e = hip_check(hipEventCreateWithFlags(&s.join, hipEventDisableTiming), "join event")) return e;
  }
  *out = &s;
  return TU_OK;
}

// `gate`, if given, is an event the first attention kernel waits for (after its stage).
int run_attention(const std::vector<AttnLaunch>& ls, int D, hipStream_t st, hipEvent_t gate = nullptr) {
  for (const auto& L : ls) {
    if (int e = hip_check(timed("rope_vt_pack", st, [&] { return launch_stage(L.rope, L.rope_tokens, L.pack, D, st); }), "RoPE/V^T pack launch")) return e;
    if (gate) {
      if (int e = hip_check(hipStreamWaitEvent(st, gate, 0), "attention gate")) return e;
      gate = nullptr;
    }
    if (int e = hip_check(timed("attention", st, [&] { return launch_attention(L.attn, L.order, D, st); }), "attention launch")) return e;
    if (L.merge_rows > 0)
      if (int e = hip_check(timed("attention_merge", st, [&] { return launch_attention_merge(L.merge, L.merge_rows, D, st); }), "merge launch")) return e;
  }
  return TU_OK;
}

// ------------------------------------------------------------------ delta plan

struct DeltaItem {
  float* state;
  const bf16_t* q;
  const bf16_t* k;
  const bf16_t* v;
  const float* beta;
  const float* g;
  float* out;
  int64_t T;
};

int plan_delta(const tu_delta_params* p, const std::vector<DeltaItem>& items, void* ws, const CallStatus& status,
               std::vector<DeltaArgs>* out, size_t* ws_bytes) {
  const int C = p->chunk, Hv = p->n_v_heads, DK = p->d_k;
  size_t max_used = 0;
  out->clear();
  for (size_t g0 = 0; g0 < items.size(); g0 += kMaxSeqPerDelta) {
    const size_t g1 = std::min(items.size(), g0 + kMaxSeqPerDelta);
    int n_active = 0;
    for (size_t i = g0; i < g1; ++i) n_active += items[i].T > 0;
    // slice d_v (16 rows of S per owner wave of the chain) into as few workgroups per
    // head as give half the CUs one (the rest serve the attention layers running
    // beside the delta layers)
    int dvs = std::min(DK, 64);
    while (dvs > 16 && (int64_t)n_active * Hv * (DK / dvs) < kCus / 2) dvs /= 2;
    DeltaArgs a{};
    a.n_k_heads = p->n_k_heads;
    a.n_v_heads = Hv;
    a.scale = p->scale;
    a.n_slices = DK / dvs;
    a.status = status;
    int chunks = 0;
    for (size_t i = g0; i < g1; ++i) {
      const auto& it = items[i];
      if (it.T <= 0) continue;
      DeltaSeq& s = a.seq[a.n_seq++];
      s.q = it.q;
      s.k = it.k;
      s.v = it.v;
      s.beta = it.beta;
      s.g = it.g;
      s.state = it.state;
      s.out = it.out;
      s.T = (int32_t)it.T;
      s.n_chunks = (int32_t)((it.T + C - 1) / C);
      s.chunk_begin = chunks;
      chunks += s.n_chunks;
    }
    a.total_chunks = chunks;
    Arena ar(ws);
    a.ws_w = static_cast<_Float16*>(ar.take(sizeof(_Float16) * (size_t)chunks * Hv * C * DK));
    a.ws_tv = static_cast<_Float16*>(ar.take(sizeof(_Float16) * (size_t)chunks * Hv * C * C));
    a.ws_p = static_cast<_Float16*>(ar.take(sizeof(_Float16) * (size_t)chunks * Hv * C * std::max(C, 32)));
    a.ws_dec = static_cast<float*>(ar.take(sizeof(float) * (size_t)chunks * Hv * 2 * C));
    a.ws_q = static_cast<_Float16*>(ar.take(sizeof(_Float16) * (size_t)chunks * p->n_k_heads * C * DK));
    a.ws_kt = static_cast<_Float16*>(ar.take(sizeof(_Float16) * (size_t)chunks * p->n_k_heads * DK * std::max(C, 32)));
    max_used = std::max(max_used, ar.used);
    if (a.n_seq > 0) out->push_back(a);
  }
  *ws_bytes = max_used;
  return TU_OK;
}

int run_delta(const std::vector<DeltaArgs>& ls, const tu_delta_params* p, hipStream_t st) {
  for (const auto& a : ls) {
    if (int e = hip_check(timed("delta_prep", st, [&] { return launch_delta_prep(a, p->d_k, p->chunk, st); }), "delta-prep launch")) return e;
    if (int e = hip_check(timed("delta_chain", st, [&] { return launch_delta_chain(a, p->d_k, p->chunk, st); }), "delta-chain launch")) return e;
  }
  return TU_OK;
}


int commit_intervals(tu_seq* s, const std::vector<tu_interval>& iv) {
  if ((int64_t)iv.size() > s->live_cap) return fail(TU_ERR_CAPACITY, "live-interval list full (%d)", s->live_cap);
  for (size_t i = 0; i < iv.size(); ++i) s->live[i] = iv[i];
  s->n_live = (int32_t)iv.size();
  return TU_OK;
}

// ------------------------------------------------------------------ key relocation

struct RelocSpan {
  int64_t row, len, delta;
};

// Rotates the keys of the rows in `spans` by their shifts in every buffer of `kbufs`
// and relabels d_pos: launches of up to kMaxRelocSpans spans x kMaxBufPerLaunch
// buffers (positions move with the first buffer group only).
int run_relocation(const std::vector<RelocSpan>& spans, const std::vector<void*>& kbufs, int32_t* d_pos,
                   const tu_attn_params* p, hipStream_t st) {
  for (size_t s0 = 0; s0 < spans.size(); s0 += kMaxRelocSpans) {
    const size_t s1 = std::min(spans.size(), s0 + kMaxRelocSpans);
    size_t b0 = 0;
    do {
      RelocArgs a{};
      a.pos = b0 == 0 ? d_pos : nullptr;
      a.n_bufs = (int32_t)std::min<size_t>(kMaxBufPerLaunch, kbufs.size() - b0);
      for (int b = 0; b < a.n_bufs; ++b) a.bufs[b] = static_cast<bf16_t*>(kbufs[b0 + b]);
      if (a.n_bufs > 0) {
        a.n_kv_heads = p->n_kv_heads;
        a.head_dim = p->head_dim;
        a.rotary_dim = p->rotary_dim;
        a.theta = p->rope_theta;
      }
      a.block_begin[0] = 0;
      for (size_t i = s0; i < s1; ++i) {
        const int k = (int)(i - s0);
        a.row[k] = (int32_t)spans[i].row;
        a.delta[k] = (int32_t)spans[i].delta;
        a.block_begin[k + 1] = a.block_begin[k] + (int32_t)spans[i].len;
      }
      a.n_spans = (int32_t)(s1 - s0);
      if (a.pos || a.n_bufs > 0)
        if (int e = hip_check(timed("relocate", st, [&] { return launch_relocate(a, st); }), "relocation launch"))
          return e;
      b0 += kMaxBufPerLaunch;
    } while (b0 < kbufs.size());
  }
  return TU_OK;
}

// The runs of `live` (row order) with the positions of each move's source range
// shifted to its destination (rows keep their place), in row order.
std::vector<tu_interval> relabel_runs(const tu_interval* live, int n_live, const int64_t* moves, int n) {
  std::vector<tu_interval> out;
  for (int i = 0; i < n_live; ++i) {
    int64_t cur = live[i].begin;
    const int64_t end = live[i].end;
    int lo = 0, hi = n;   // first move whose source ends after cur
    while (lo < hi) {
      const int mid = (lo + hi) / 2;
      if (moves[3 * mid + 1] <= cur) lo = mid + 1;
      else hi = mid;
    }
    for (int q = lo; q < n && moves[3 * q] < end; ++q) {
      const int64_t a = std::max(cur, moves[3 * q]), b = std::min(end, moves[3 * q + 1]);
      const int64_t d = moves[3 * q + 2] - moves[3 * q];
      push_run(out, cur, a);
      push_run(out, a + d, b + d);
      cur = b;
    }
    push_run(out, cur, end);
  }
  return out;
}

// ------------------------------------------------------------------ stack update

struct StackPlan {
  std::vector<RangeCheck> rc;
  std::vector<std::vector<tu_interval>> final_iv;   // after the tail is appended
  std::vector<int64_t> cursor_after;                // cursor once the update commits
  std::vector<int64_t> tail_begin;   // row offset of each context in the packed tail inputs
  // removal of rows inside the tail once it is prefilled (maintenance delimiters)
  std::vector<RangeCheck> post_rc;
  std::vector<tu_seq> post_seq;      // each context as it stands after the append
  bool any_post = false;
  int n_attn = 0, n_delta = 0;
};

int validate_stack(const tu_update* u, StackPlan* sp) {
  if (!u) return fail(TU_ERR_ARG, "null update");
  if (u->n_seq < 0 || (u->n_seq > 0 && !u->seqs)) return fail(TU_ERR_ARG, "bad context list");
  if (u->n_layers < 0 || (u->n_layers > 0 && !u->layers)) return fail(TU_ERR_ARG, "bad layer list");
  sp->rc.assign(u->n_seq, RangeCheck{});
  sp->final_iv.assign(u->n_seq, {});
  sp->cursor_after.assign(u->n_seq, 0);
  sp->tail_begin.assign(u->n_seq + 1, 0);
  sp->post_rc.assign(u->n_seq, RangeCheck{});
  sp->post_seq.assign(u->n_seq, tu_seq{});
  sp->any_post = false;
  for (int l = 0; l < u->n_layers; ++l) {
    const int kind = u->layers[l].kind;
    if (kind == TU_LAYER_ATTN) ++sp->n_attn;
    else if (kind == TU_LAYER_DELTA) ++sp->n_delta;
    else return fail(TU_ERR_ARG, "layer %d: unknown kind %d", l, kind);
  }
  if (sp->n_attn) if (int e = check_attn(&u->attn)) return e;
  if (sp->n_delta) if (int e = check_delta(&u->delta)) return e;
  for (int s = 0; s < u->n_seq; ++s) {
    const tu_seq_update& su = u->seqs[s];
    if (int e = check_seq(su.seq)) return e;
    for (int t = 0; t < s; ++t)
      if (u->seqs[t].seq == su.seq) return fail(TU_ERR_ARG, "context %d appears twice", s);
    if (su.T < 0) return fail(TU_ERR_ARG, "context %d: negative T", s);
    if (int e = check_ranges(su.seq, su.ranges, su.n_ranges, &sp->rc[s])) return e;
    const int64_t L_keep = su.seq->len - sp->rc[s].removed;
    if (L_keep + su.T > su.seq->capacity)
      return fail(TU_ERR_CAPACITY, "context %d: %lld surviving + %lld tail rows exceed capacity %lld", s,
                  (long long)L_keep, (long long)su.T, (long long)su.seq->capacity);
    if (L_keep + su.T > INT32_MAX / 2) return fail(TU_ERR_ARG, "context %d: too many rows", s);
    const int pl = su.placement;
    if (pl != TU_PLACE_TAIL && pl != TU_PLACE_SLOT && pl != TU_PLACE_RELOCATE)
      return fail(TU_ERR_ARG, "context %d: unknown placement %d", s, pl);
    // the tail is computed at next_pos + i unless it is slot-placed
    if (pl != TU_PLACE_SLOT && su.seq->next_pos + su.T > INT32_MAX)
      return fail(TU_ERR_ARG, "context %d: positions overflow int32", s);
    sp->final_iv[s] = sp->rc[s].live_after;
    if (pl == TU_PLACE_TAIL) {
      if (su.n_place_runs != 0) return fail(TU_ERR_ARG, "context %d: placement runs given for a true-tail update", s);
      push_run(sp->final_iv[s], su.seq->next_pos, su.seq->next_pos + su.T);
      sp->cursor_after[s] = su.seq->next_pos + su.T;
    } else {
      if (int e = check_place_runs(su.place_runs, su.n_place_runs, su.T, sp->rc[s].live_after, s)) return e;
      int64_t last = 0;
      for (int q = 0; q < su.n_place_runs; ++q) {
        push_run(sp->final_iv[s], su.place_runs[2 * q], su.place_runs[2 * q + 1]);
        last = std::max(last, su.place_runs[2 * q + 1]);
      }
      sp->cursor_after[s] = std::max(pl == TU_PLACE_SLOT ? su.seq->next_pos : su.seq->next_pos + su.T, last);
    }
    if ((int64_t)sp->final_iv[s].size() > su.seq->live_cap)
      return fail(TU_ERR_CAPACITY, "context %d: live-interval list would exceed %d", s, su.seq->live_cap);
    // ranges removed after the prefill must be made of this call's tail positions
    tu_seq& ps = sp->post_seq[s];
    ps = *su.seq;
    ps.len = L_keep + su.T;
    ps.next_pos = sp->cursor_after[s];
    ps.live = sp->final_iv[s].data();
    ps.n_live = (int32_t)sp->final_iv[s].size();
    if (su.n_post_ranges < 0 || (su.n_post_ranges > 0 && !su.post_ranges))
      return fail(TU_ERR_ARG, "context %d: bad post-prefill ranges", s);
    if (int e = check_ranges(&ps, su.post_ranges, su.n_post_ranges, &sp->post_rc[s])) return e;
    for (const auto& span : sp->post_rc[s].spans)
      if (span.first < L_keep)
        return fail(TU_ERR_RANGE, "context %d: a post-prefill range holds positions outside this call's tail", s);
    if ((int64_t)sp->post_rc[s].live_after.size() > su.seq->live_cap)
      return fail(TU_ERR_CAPACITY, "context %d: live-interval list would exceed %d", s, su.seq->live_cap);
    sp->any_post = sp->any_post || sp->post_rc[s].removed > 0;
    sp->tail_begin[s + 1] = sp->tail_begin[s] + su.T;
  }
  const int64_t total_T = sp->tail_begin[u->n_seq];
  for (int l = 0; l < u->n_layers; ++l) {
    const tu_layer_io& L = u->layers[l];
    if (total_T > 0) {
      if (!L.q || !L.k || !L.v || !L.out) return fail(TU_ERR_ARG, "layer %d: null tail tensor", l);
      if (!aligned16(L.q) || !aligned16(L.k) || !aligned16(L.v) || !aligned16(L.out))
        return fail(TU_ERR_ARG, "layer %d: tail tensors must be 16-byte aligned", l);
    }
    if (L.kind == TU_LAYER_ATTN) {
      if (u->n_seq > 0 && (!L.k_cache || !L.v_cache)) return fail(TU_ERR_ARG, "layer %d: null cache list", l);
      for (int s = 0; s < u->n_seq; ++s) {
        if (u->seqs[s].seq->capacity == 0) continue;
        if (!L.k_cache[s] || !L.v_cache[s]) return fail(TU_ERR_ARG, "layer %d context %d: null cache", l, s);
        if (!aligned16(L.k_cache[s]) || !aligned16(L.v_cache[s]))
          return fail(TU_ERR_ARG, "layer %d context %d: caches must be 16-byte aligned", l, s);
      }
    } else {
      if (total_T > 0 && (!L.beta || !L.g)) return fail(TU_ERR_ARG, "layer %d: null beta/g", l);
      if (u->n_seq > 0 && !L.state) return fail(TU_ERR_ARG, "layer %d: null state list", l);
      for (int s = 0; s < u->n_seq; ++s) {
        if (!L.state[s]) return fail(TU_ERR_ARG, "layer %d context %d: null state", l, s);
        if (!aligned16(L.state[s])) return fail(TU_ERR_ARG, "layer %d context %d: state must be 16-byte aligned", l, s);
      }
    }
  }
  return TU_OK;
}

// Rows of the tail removed once it is prefilled: a second compaction of every
// attention layer, against each context as it stands after the append (no keep-scan:
// nothing reads its index list, and the tail positions were just written).
std::vector<CompactItem> stack_post_items(const tu_update* u, StackPlan& sp) {
  std::vector<CompactItem> items;
  for (int s = 0; s < u->n_seq; ++s) {
    const tu_seq_update& su = u->seqs[s];
    if (sp.post_rc[s].removed == 0) continue;
    CompactItem it;
    it.seq = &sp.post_seq[s];
    it.ranges = su.post_ranges;
    it.n_ranges = su.n_post_ranges;
    it.rc = sp.post_rc[s];
    it.src_index = nullptr;
    it.scan = false;
    for (int l = 0; l < u->n_layers; ++l)
      if (u->layers[l].kind == TU_LAYER_ATTN) {
        it.bufs.push_back(u->layers[l].k_cache[s]);
        it.bufs.push_back(u->layers[l].v_cache[s]);
      }
    items.push_back(it);
  }
  return items;
}

std::vector<CompactItem> stack_compact_items(const tu_update* u, const StackPlan& sp) {
  std::vector<CompactItem> items;
  for (int s = 0; s < u->n_seq; ++s) {
    const tu_seq_update& su = u->seqs[s];
    CompactItem it;
    it.seq = su.seq;
    it.ranges = su.ranges;
    it.n_ranges = su.n_ranges;
    it.rc = sp.rc[s];
    it.src_index = su.src_index;
    for (int l = 0; l < u->n_layers; ++l)
      if (u->layers[l].kind == TU_LAYER_ATTN) {
        it.bufs.push_back(u->layers[l].k_cache[s]);
        it.bufs.push_back(u->layers[l].v_cache[s]);
      }
    items.push_back(std::move(it));
  }
  return items;
}

std::vector<AttnItem> stack_attn_items(const tu_update* u, const StackPlan& sp, const tu_layer_io& L) {
  std::vector<AttnItem> items;
  const int64_t qrow = (int64_t)u->attn.n_q_heads * u->attn.head_dim;
  const int64_t krow = (int64_t)u->attn.n_kv_heads * u->attn.head_dim;
  for (int s = 0; s < u->n_seq; ++s) {
    const tu_seq_update& su = u->seqs[s];
    AttnItem it;
    it.seq = su.seq;
    it.L_keep = su.seq->len - sp.rc[s].removed;
    it.T = su.T;
    it.cursor = su.seq->next_pos;
    it.k_cache = L.k_cache ? L.k_cache[s] : nullptr;
    it.v_cache = L.v_cache ? L.v_cache[s] : nullptr;
    const int64_t r0 = sp.tail_begin[s];
    it.q = static_cast<const bf16_t*>(L.q) + r0 * qrow;
    it.k = static_cast<const bf16_t*>(L.k) + r0 * krow;
    it.v = static_cast<const bf16_t*>(L.v) + r0 * krow;
    it.out = L.out + r0 * qrow;
    it.q_hat = nullptr;
    it.vt_cache = L.vt_cache ? L.vt_cache[s] : nullptr;
    // rows of the copy still current: up to the first row this update's removal moves
    it.vt_rows = std::min(su.seq->vt_rows, sp.rc[s].removed > 0 ? sp.rc[s].first_row : su.seq->len);
    if (su.placement == TU_PLACE_SLOT) {
      it.place_runs = su.place_runs;
      it.n_place_runs = su.n_place_runs;
    }
    items.push_back(it);
  }
  return items;
}

// The (attention layer, context) items of the attention layers in groups that share a set
// of launches. A layer whose own workgroups (before key splits) fill the chip's CUs keeps
// a set of its own: its launch already runs whole waves, and mixing layers of that size
// spreads the dies over more key/value streams at once. All smaller layers share one set,
// so a deep stack of short tails runs as a few launches whose splits fill the chip.
std::vector<std::vector<AttnItem>> stack_attn_groups(const tu_update* u, const StackPlan& sp) {
  std::vector<std::vector<AttnItem>> groups;
  std::vector<AttnItem> small;
  const int G = u->attn.n_q_heads / u->attn.n_kv_heads;
  for (int l = 0; l < u->n_layers; ++l) {
    if (u->layers[l].kind != TU_LAYER_ATTN) continue;
    auto items = stack_attn_items(u, sp, u->layers[l]);
    int64_t wg = 0;
    for (const auto& it : items) wg += (int64_t)u->attn.n_kv_heads * ((it.T * G + kAttnRows - 1) / kAttnRows);
    if (wg >= kCus)
      groups.push_back(std::move(items));
    else
      small.insert(small.end(), items.begin(), items.end());
  }
  if (!small.empty()) groups.push_back(std::move(small));
  return groups;
}

void append_delta_items(const tu_update* u, const StackPlan& sp, const tu_layer_io& L,
                        std::vector<DeltaItem>* items) {
  const int64_t krow = (int64_t)u->delta.n_k_heads * u->delta.d_k;
  const int64_t vrow = (int64_t)u->delta.n_v_heads * u->delta.d_v;
  for (int s = 0; s < u->n_seq; ++s) {
    const int64_t r0 = sp.tail_begin[s];
    DeltaItem it;
    it.state = L.state[s];
    it.q = static_cast<const bf16_t*>(L.q) + r0 * krow;
    it.k = static_cast<const bf16_t*>(L.k) + r0 * krow;
    it.v = static_cast<const bf16_t*>(L.v) + r0 * vrow;
    it.beta = L.beta + r0 * u->delta.n_v_heads;
    it.g = L.g + r0 * u->delta.n_v_heads;
    it.out = L.out + r0 * vrow;
    it.T = u->seqs[s].T;
    items->push_back(it);
  }
}

// Items of every delta layer of the stack, layer by layer and context by context.
// Each (layer, context) pair owns its state and its inputs, so all of them are
// independent and share launches (up to kMaxSeqPerDelta items each).
std::vector<DeltaItem> stack_delta_items(const tu_update* u, const StackPlan& sp) {
  std::vector<DeltaItem> items;
  for (int l = 0; l < u->n_layers; ++l) {
    const tu_layer_io& L = u->layers[l];
    if (L.kind != TU_LAYER_DELTA) continue;
    append_delta_items(u, sp, L, &items);
  }
  return items;
}

}  // namespace
}  // namespace tu

using namespace tu;

extern "C" {

int tu_abi_version(void) { return TU_ABI_VERSION; }

const char* tu_last_error(void) { return g_err.c_str(); }

static_assert(TU_FAULT_POSITIONS == tu::kFaultPositions && TU_FAULT_WAIT == tu::kFaultWait &&
                  TU_FAULT_RANGE == tu::kFaultRange, "fault bits");

int tu_workspace_faults(const void* workspace, int32_t* faults, void* stream) {
  if (!faults || !workspace) return fail(TU_ERR_ARG, "null workspace or faults");
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint64_t block[(kStatusLastOffset + 8) / 8] = {};
  if (int e = hip_check(hipMemcpyAsync(block, workspace, sizeof(block), hipMemcpyDeviceToHost, st),
                        "reading the status words"))
    return e;
  if (int e = hip_check(hipStreamSynchronize(st), "stream synchronise")) return e;
  const uint64_t word = block[0];
  const uint32_t last = (uint32_t)block[kStatusLastOffset / 8];
  *faults = (uint32_t)(word >> 32) == last ? (int32_t)(uint32_t)word : 0;
  return ok();
}

int tu_validate_ranges(const tu_seq* seq, const int64_t* ranges, int32_t n_ranges, int64_t* n_removed) {
  if (int e = check_seq(seq)) return e;
  RangeCheck rc;
  if (int e = check_ranges(seq, ranges, n_ranges, &rc)) return e;
  if (n_removed) *n_removed = rc.removed;
  return ok();
}

size_t compact_kv_workspace_size(int64_t len, int32_t n_layers, int32_t n_kv_heads, int32_t head_dim) {
  if (len < 0 || n_layers < 0 || n_kv_heads <= 0 || head_dim <= 0) return 0;
  const int row_bytes = n_kv_heads * head_dim * 2;
  if (row_bytes > kGatherStripeBytes) return 0;
  // the worst case: every row behind the first one moves
  tu_seq fake{};
  fake.len = len;
  std::vector<CompactItem> items(1);
  items[0].seq = &fake;
  items[0].n_ranges = 0;   // sizing only: spans are not read
  items[0].rc.removed = 1;
  items[0].rc.first_row = 0;
  items[0].src_index = nullptr;
  items[0].bufs.assign(2 * (size_t)n_layers, nullptr);
  fake.len = len + 1;
  CompactPlan plan;
  plan_compaction(items, row_bytes, nullptr, CallStatus{}, &plan);
  return kStatusBytes + plan.ws_bytes;
}

}  // extern "C"

// Fixed scratch of compact_kv_noalloc: each GPU the library runs on holds one copy until
// the process ends. In host code its name is a stand-in, not a device address; the
// address comes from hipGetSymbolAddress, once per device, with that device current.
static __device__ __align__(256) char scratch[TU_NOALLOC_SCRATCH_BYTES];

namespace tu {
namespace {

std::mutex g_scratch_mutex;
void* g_scratch_ptr[64] = {};

int scratch_of_current_device(void** out) {
  int dev = 0;
  if (int e = hip_check(hipGetDevice(&dev), "current device")) return e;
  if (dev < 0 || dev >= 64) return fail(TU_ERR_HIP, "device index %d out of range", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (int e = hip_check(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "scratch address")) return e;
    if (!p) return fail(TU_ERR_HIP, "no scratch address on device %d", dev);
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return TU_OK;
}

}  // namespace
}  // namespace tu

namespace tu {
namespace {

// compact_kv with the workspace [base, base + bytes), or (use_scratch) the fixed scratch
// of the current device, whose address is fetched once the host checks passed: status
// block first, unless `status` names a block of its own (then the whole range is the
// compaction's).
int compact_with(tu_seq* seq, void* const* k_layers, void* const* v_layers, int32_t n_layers, int32_t n_kv_heads,
                 int32_t head_dim, const int64_t* ranges, int32_t n_ranges, int32_t* src_index, void* base,
                 size_t bytes, bool use_scratch, void* status, const char* space, hipStream_t st) {
  if (int e = check_seq(seq)) return e;
  if (n_layers < 0 || (n_layers > 0 && (!k_layers || !v_layers))) return fail(TU_ERR_ARG, "bad layer arrays");
  if (n_kv_heads <= 0 || head_dim <= 0 || ((long)n_kv_heads * head_dim * 2) % 16)
    return fail(TU_ERR_ARG, "cache rows must be a positive multiple of 16 bytes");
  const int row_bytes = n_kv_heads * head_dim * 2;
  if (row_bytes > kGatherStripeBytes || (row_bytes < 128 && 128 % row_bytes) || (row_bytes > 128 && row_bytes % 128))
    return fail(TU_ERR_ARG, "unsupported cache row size %d bytes", row_bytes);
  for (int l = 0; l < n_layers; ++l) {
    if (!k_layers[l] || !v_layers[l]) return fail(TU_ERR_ARG, "null cache of layer %d", l);
    if (!aligned16(k_layers[l]) || !aligned16(v_layers[l])) return fail(TU_ERR_ARG, "caches must be 16-byte aligned");
  }
  std::vector<CompactItem> items(1);
  items[0].seq = seq;
  items[0].ranges = ranges;
  items[0].n_ranges = n_ranges;
  items[0].src_index = src_index;
  if (int e = check_ranges(seq, ranges, n_ranges, &items[0].rc)) return e;
  if ((int64_t)items[0].rc.live_after.size() > seq->live_cap)
    return fail(TU_ERR_CAPACITY, "live-interval list would exceed %d", seq->live_cap);
  for (int l = 0; l < n_layers; ++l) {
    items[0].bufs.push_back(k_layers[l]);
    items[0].bufs.push_back(v_layers[l]);
  }
  CompactPlan plan;
  plan_compaction(items, row_bytes, nullptr, CallStatus{}, &plan);
  const size_t need = (status ? 0 : kStatusBytes) + plan.ws_bytes;
  if (bytes < need) return fail(TU_ERR_WORKSPACE, "%s of %zu bytes, %zu needed", space, bytes, need);
  if (use_scratch)
    if (int e = scratch_of_current_device(&base)) return e;
  if (!base) return fail(TU_ERR_WORKSPACE, "null %s", space);
  if (!aligned16(base) || (status && !aligned16(status)))
    return fail(TU_ERR_WORKSPACE, "%s and status must be 16-byte aligned", space);
  items[0].src_index = src_index;
  const CallStatus cs = call_status(status ? status : base);
  if (int e = plan_compaction(items, row_bytes, status ? base : after_status(base), cs, &plan)) return e;
  const uint64_t launches = g_launches;
  if (int e = run_compaction(plan, st)) return e;
  if (g_launches == launches)   // nothing to move or scan: record the call all the same
    if (int e = hip_check(launch_status_mark(cs, st), "status mark")) return e;
  const int64_t removed = items[0].rc.removed;
  commit_intervals(seq, items[0].rc.live_after);
  seq->len -= removed;
  if (removed > 0) seq->vt_rows = std::min(seq->vt_rows, items[0].rc.first_row);
  return ok();
}

}  // namespace
}  // namespace tu

extern "C" {

int compact_kv(tu_seq* seq, void* const* k_layers, void* const* v_layers, int32_t n_layers, int32_t n_kv_heads,
               int32_t head_dim, const int64_t* ranges, int32_t n_ranges, int32_t* src_index, void* workspace,
               size_t workspace_bytes, void* stream) {
  return compact_with(seq, k_layers, v_layers, n_layers, n_kv_heads, head_dim, ranges, n_ranges, src_index, workspace,
                      workspace_bytes, false, nullptr, "workspace", static_cast<hipStream_t>(stream));
}

int compact_kv_noalloc(tu_seq* seq, void* const* k_layers, void* const* v_layers, int32_t n_layers,
                       int32_t n_kv_heads, int32_t head_dim, const int64_t* ranges, int32_t n_ranges,
                       int32_t* src_index, void* status, void* stream) {
  return compact_with(seq, k_layers, v_layers, n_layers, n_kv_heads, head_dim, ranges, n_ranges, src_index, nullptr,
                      TU_NOALLOC_SCRATCH_BYTES, true, status, "the fixed scratch", static_cast<hipStream_t>(stream));
}

size_t tail_prefill_attention_workspace_size(const tu_attn_params* p, int64_t T, int64_t len) {
  if (check_attn(p) || T < 0 || len < 0) return 0;
  tu_seq fake{};
  std::vector<AttnItem> items(1);
  items[0] = AttnItem{&fake, len, T, 0, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  std::vector<AttnLaunch> ls;
  size_t bytes = 0;
  plan_attention(p, items, nullptr, CallStatus{}, &ls, &bytes);
  return kStatusBytes + bytes;
}

size_t tu_vt_cache_bytes(int64_t capacity, int32_t n_kv_heads, int32_t head_dim) {
  if (capacity < 0 || n_kv_heads <= 0 || (head_dim != 64 && head_dim != 128 && head_dim != 256)) return 0;
  return sizeof(_Float16) * (size_t)n_kv_heads * (size_t)vt_head_tiles(capacity) * head_dim * kVtRow;
}

int refresh_vt_cache(tu_seq* seq, void* const* v_layers, void* const* vt_layers, int32_t n_layers, int32_t n_kv_heads,
                     int32_t head_dim, void* workspace, size_t workspace_bytes, void* stream) {
  if (int e = check_seq(seq)) return e;
  if (n_layers < 0 || n_layers > kMaxSeqPerLaunch || (n_layers > 0 && (!v_layers || !vt_layers)))
    return fail(TU_ERR_ARG, "0 .. %d layers with value caches and V^T copies", kMaxSeqPerLaunch);
  if (tu_vt_cache_bytes(seq->capacity, n_kv_heads, head_dim) == 0 && seq->capacity > 0)
    return fail(TU_ERR_ARG, "unsupported head shape");
  for (int l = 0; l < n_layers; ++l)
    if (!v_layers[l] || !vt_layers[l] || !aligned16(v_layers[l]) || !aligned16(vt_layers[l]))
      return fail(TU_ERR_ARG, "layer %d: null or misaligned buffer", l);
  if (!workspace || workspace_bytes < kStatusBytes)
    return fail(TU_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes, kStatusBytes);
  if (!aligned16(workspace)) return fail(TU_ERR_WORKSPACE, "workspace must be 16-byte aligned");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const CallStatus cs = call_status(workspace);
  const int begin = (int)(std::min(seq->vt_rows, seq->len) / kAttnKeys);
  const int end = (int)vt_head_tiles(seq->len);
  if (n_layers > 0 && end > begin) {
    // the stage kernel with packing workgroups only: one entry per layer, all with no tail
    RopeArgs r{};
    PackArgs pk{};
    r.n_kv_heads = n_kv_heads;
    r.head_dim = head_dim;
    for (int l = 0; l < n_layers; ++l) {
      RopeSeq& rs = r.seq[r.n_seq++];
      rs.v_cache = static_cast<bf16_t*>(v_layers[l]);
      rs.v = rs.v_cache;
      rs.L_keep = (int32_t)seq->len;
      rs.T = 0;
      PackSeq& ps = pk.seq[pk.n_seq++];
      ps.vt = static_cast<_Float16*>(vt_layers[l]);
      ps.tile_begin = begin;
      ps.tile_end = end;
      ps.head_tiles = (int)vt_head_tiles(seq->capacity);
      ps.pack_begin = pk.pack_items;
      pk.pack_items += n_kv_heads * (end - begin);
    }
    pk.status = cs;
    if (int e = hip_check(timed("rope_vt_pack", st, [&] { return launch_stage(r, 0, pk, head_dim, st); }),
                          "V^T pack launch"))
      return e;
  } else if (int e = hip_check(launch_status_mark(cs, st), "status mark")) {
    return e;
  }
  seq->vt_rows = seq->len;
  return ok();
}

int tail_prefill_attention(const tu_seq* seq, void* k_cache, void* v_cache, void* vt_cache, const tu_attn_params* p,
                           const void* q, const void* k, const void* v, int64_t T, float* out, void* q_hat,
                           void* workspace, size_t workspace_bytes, void* stream) {
  if (int e = check_seq(seq)) return e;
  if (int e = check_attn(p)) return e;
  if (T < 0) return fail(TU_ERR_ARG, "negative T");
  if (seq->len + T > seq->capacity)
    return fail(TU_ERR_CAPACITY, "%lld rows + %lld tail rows exceed capacity %lld", (long long)seq->len, (long long)T,
                (long long)seq->capacity);
  if (seq->next_pos + T > INT32_MAX) return fail(TU_ERR_ARG, "positions overflow int32");
  if (T == 0) return ok();
  if (!k_cache || !v_cache || !q || !k || !v || !out) return fail(TU_ERR_ARG, "null tensor");
  if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(q) || !aligned16(k) || !aligned16(v) ||
      !aligned16(out) || (q_hat && !aligned16(q_hat)) || (vt_cache && !aligned16(vt_cache)))
    return fail(TU_ERR_ARG, "tensors must be 16-byte aligned");
  std::vector<AttnItem> items(1);
  items[0] = AttnItem{seq, seq->len, T, seq->next_pos, k_cache, v_cache, static_cast<const bf16_t*>(q),
                      static_cast<const bf16_t*>(k), static_cast<const bf16_t*>(v), out,
                      static_cast<bf16_t*>(q_hat)};
  items[0].vt_cache = vt_cache;
  items[0].vt_rows = seq->vt_rows;
  std::vector<AttnLaunch> ls;
  size_t need = 0;
  plan_attention(p, items, nullptr, CallStatus{}, &ls, &need);
  need += kStatusBytes;
  if (!workspace || workspace_bytes < need)
    return fail(TU_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
  if (!aligned16(workspace)) return fail(TU_ERR_WORKSPACE, "workspace must be 16-byte aligned");
  hipStream_t st = static_cast<hipStream_t>(stream);
  plan_attention(p, items, after_status(workspace), call_status(workspace), &ls, &need);
  if (int e = run_attention(ls, p->head_dim, st)) return e;
  return ok();
}

int commit_tail(tu_seq* seq, int64_t T) {
  if (int e = check_seq(seq)) return e;
  if (T < 0) return fail(TU_ERR_ARG, "negative T");
  if (seq->len + T > seq->capacity) return fail(TU_ERR_CAPACITY, "commit exceeds capacity");
  if (seq->next_pos + T > INT32_MAX) return fail(TU_ERR_ARG, "positions overflow int32");
  std::vector<tu_interval> iv(seq->live, seq->live + seq->n_live);
  push_run(iv, seq->next_pos, seq->next_pos + T);
  if ((int64_t)iv.size() > seq->live_cap) return fail(TU_ERR_CAPACITY, "live-interval list full");
  commit_intervals(seq, iv);
  seq->len += T;
  seq->next_pos += T;
  seq->vt_rows = seq->len;
  return ok();
}

size_t delta_rule_continue_workspace_size(const tu_delta_params* p, int64_t T) {
  if (check_delta(p) || T < 0) return 0;
  std::vector<DeltaItem> items(1);
  items[0] = DeltaItem{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, T};
  std::vector<DeltaArgs> ls;
  size_t bytes = 0;
  plan_delta(p, items, nullptr, CallStatus{}, &ls, &bytes);
  return kStatusBytes + bytes;
}

int delta_rule_continue(float* state, const void* q, const void* k, const void* v, const float* beta, const float* g,
                        int64_t T, const tu_delta_params* p, float* out, void* workspace, size_t workspace_bytes,
                        void* stream) {
  if (int e = check_delta(p)) return e;
  if (T < 0) return fail(TU_ERR_ARG, "negative T");
  if (T == 0) return ok();
  if (T > INT32_MAX / 2) return fail(TU_ERR_ARG, "T too large");
  if (!state || !q || !k || !v || !beta || !g || !out) return fail(TU_ERR_ARG, "null tensor");
  if (!aligned16(state) || !aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
    return fail(TU_ERR_ARG, "tensors must be 16-byte aligned");
  std::vector<DeltaItem> items(1);
  items[0] = DeltaItem{state, static_cast<const bf16_t*>(q), static_cast<const bf16_t*>(k),
                       static_cast<const bf16_t*>(v), beta, g, out, T};
  std::vector<DeltaArgs> ls;
  size_t need = 0;
  plan_delta(p, items, nullptr, CallStatus{}, &ls, &need);
  need += kStatusBytes;
  if (!workspace || workspace_bytes < need)
    return fail(TU_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
  if (!aligned16(workspace)) return fail(TU_ERR_WORKSPACE, "workspace must be 16-byte aligned");
  hipStream_t st = static_cast<hipStream_t>(stream);
  plan_delta(p, items, after_status(workspace), call_status(workspace), &ls, &need);
  if (int e = run_delta(ls, p, st)) return e;
  return ok();
}

int short_conv_continue_batch(const tu_conv_tensor* tensors, int32_t n, int32_t width, int32_t activation,
                              void* stream) {
  if (n < 0 || (n > 0 && !tensors)) return fail(TU_ERR_ARG, "bad tensor array");
  if (width < 1 || width > 8) return fail(TU_ERR_ARG, "width must be 1 .. 8");
  if (activation != TU_CONV_IDENTITY && activation != TU_CONV_SILU) return fail(TU_ERR_ARG, "unknown activation");
  for (int i = 0; i < n; ++i) {
    const tu_conv_tensor& t = tensors[i];
    if (t.T < 0) return fail(TU_ERR_ARG, "tensor %d: negative T", i);
    if (t.T > INT32_MAX / 2) return fail(TU_ERR_ARG, "tensor %d: T too large", i);
    if (t.channels <= 0 || t.channels % 8) return fail(TU_ERR_ARG, "tensor %d: channels must be a positive multiple of 8", i);
    if (t.T == 0) continue;
    if (!t.x || !t.weight || !t.out || (width > 1 && !t.state)) return fail(TU_ERR_ARG, "tensor %d: null pointer", i);
    if (!aligned16(t.x) || !aligned16(t.weight) || !aligned16(t.out) || (t.state && !aligned16(t.state)))
      return fail(TU_ERR_ARG, "tensor %d: pointers must be 16-byte aligned", i);
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  ConvArgs a{};
  int blocks = 0;
  auto flush = [&]() -> int {
    if (a.n_jobs == 0) return TU_OK;
    if (int e = hip_check(timed("short_conv", st, [&] { return launch_short_conv(a, blocks, width, st); }),
                          "short-conv launch"))
      return e;
    a = ConvArgs{};
    blocks = 0;
    return TU_OK;
  };
  for (int i = 0; i < n; ++i) {
    const tu_conv_tensor& t = tensors[i];
    if (t.T == 0) continue;
    ConvJob& j = a.job[a.n_jobs++];
    j.state = static_cast<bf16_t*>(t.state);
    j.x = static_cast<const bf16_t*>(t.x);
    j.w = static_cast<const bf16_t*>(t.weight);
    j.out = static_cast<bf16_t*>(t.out);
    j.T = (int32_t)t.T;
    j.C = t.channels;
    j.act = activation == TU_CONV_SILU;
    blocks += conv_blocks(j, blocks);
    if (a.n_jobs == kMaxConvJobs)
      if (int e = flush()) return e;
  }
  if (int e = flush()) return e;
  return ok();
}

int short_conv_continue(void* state, const void* x, const void* weight, int64_t T, int32_t channels, int32_t width,
                        int32_t activation, void* out, void* stream) {
  const tu_conv_tensor t{state, x, weight, out, T, channels, 0};
  return short_conv_continue_batch(&t, 1, width, activation, stream);
}

}  // extern "C"

namespace {

// Workspace of a stack update: [compaction / attention region | delta region]. Delta
// layers run on a second stream concurrently with the attention path, so the two
// regions are disjoint. Attention layers run in order and reuse their region; the
// (layer, context) items of all delta layers are planned together into launches of
// up to kMaxSeqPerDelta items, which run in order and reuse the delta region.
struct StackWorkspace {
  size_t attn = 0;    // compaction and attention layers
  size_t delta = 0;   // delta layers
  size_t total() const { return kStatusBytes + align_up(attn) + align_up(delta); }
};

StackWorkspace stack_workspace(const tu_update* u, StackPlan& sp) {
  StackWorkspace w;
  w.attn = kAlign;
  if (sp.n_attn) {
    auto items = stack_compact_items(u, sp);
    CompactPlan cp;
    plan_compaction(items, u->attn.n_kv_heads * u->attn.head_dim * 2, nullptr, CallStatus{}, &cp);
    w.attn = std::max(w.attn, cp.ws_bytes);
    if (sp.any_post) {
      auto post = stack_post_items(u, sp);
      plan_compaction(post, u->attn.n_kv_heads * u->attn.head_dim * 2, nullptr, CallStatus{}, &cp);
      w.attn = std::max(w.attn, cp.ws_bytes);
    }
  }
  for (auto& items : stack_attn_groups(u, sp)) {
    size_t b = 0;
    std::vector<AttnLaunch> ls;
    plan_attention(&u->attn, items, nullptr, CallStatus{}, &ls, &b);
    w.attn = std::max(w.attn, b);
  }
  auto items = stack_delta_items(u, sp);
  if (!items.empty()) {
    std::vector<DeltaArgs> ls;
    plan_delta(&u->delta, items, nullptr, CallStatus{}, &ls, &w.delta);
  }
  return w;
}

}  // namespace

extern "C" {

size_t update_layer_stack_workspace_size(const tu_update* u) {
  StackPlan sp;
  if (validate_stack(u, &sp)) return 0;
  return stack_workspace(u, sp).total();
}

int relocate_keys(tu_seq* seq, void* const* k_layers, int32_t n_layers, const tu_attn_params* p,
                  const int64_t* moves, int32_t n_moves, void* stream) {
  if (int e = check_seq(seq)) return e;
  if (n_layers < 0 || (n_layers > 0 && !k_layers)) return fail(TU_ERR_ARG, "bad layer array");
  if (n_layers > 0) {
    if (int e = check_attn(p)) return e;
    for (int l = 0; l < n_layers; ++l)
      if (!k_layers[l] || !aligned16(k_layers[l])) return fail(TU_ERR_ARG, "key cache %d null or misaligned", l);
  }
  if (n_moves < 0 || n_moves > TU_MAX_RANGES || (n_moves > 0 && !moves))
    return fail(TU_ERR_ARG, "0 .. %d moves", TU_MAX_RANGES);
  const RunIndex ri(seq->live, seq->n_live);
  std::vector<int64_t> src(2 * (size_t)std::max(1, (int)n_moves));
  std::vector<RelocSpan> spans;
  std::vector<tu_interval> dst;
  int64_t prev_end = INT64_MIN, last = seq->next_pos;
  for (int q = 0; q < n_moves; ++q) {
    const int64_t s = moves[3 * q], e = moves[3 * q + 1], d = moves[3 * q + 2];
    if (e <= s || s < prev_end || s < 0)
      return fail(TU_ERR_RANGE, "move %d: sources must be non-empty, sorted and disjoint", q);
    if (d < 0 || d + (e - s) > INT32_MAX) return fail(TU_ERR_RANGE, "move %d: destination outside [0, 2^31 - 1)", q);
    std::vector<std::pair<int64_t, int64_t>> sp;
    if (!range_rows(ri, s, e, &sp)) return fail(TU_ERR_RANGE, "move %d: source [%lld,%lld) is not live", q,
                                               (long long)s, (long long)e);
    for (const auto& x : sp)
      if (d != s) spans.push_back({x.first, x.second, d - s});
    src[2 * q] = s;
    src[2 * q + 1] = e;
    dst.push_back({d, d + (e - s)});
    last = std::max(last, d + (e - s));
    prev_end = e;
  }
  if ((int)spans.size() > TU_MAX_RANGES) return fail(TU_ERR_RANGE, "the moves map to more than %d row spans", TU_MAX_RANGES);
  // destinations: disjoint from each other and from every row that stays
  std::vector<tu_interval> all = subtract_runs(seq->live, seq->n_live, src.data(), n_moves);
  all.insert(all.end(), dst.begin(), dst.end());
  std::sort(all.begin(), all.end(), [](const tu_interval& x, const tu_interval& y) { return x.begin < y.begin; });
  for (size_t i = 1; i < all.size(); ++i)
    if (all[i].begin < all[i - 1].end) return fail(TU_ERR_RANGE, "destinations overlap each other or live rows");
  const std::vector<tu_interval> runs = relabel_runs(seq->live, seq->n_live, moves, n_moves);
  if ((int64_t)runs.size() > seq->live_cap) return fail(TU_ERR_CAPACITY, "live-interval list would exceed %d", seq->live_cap);
  std::vector<void*> kbufs(k_layers, k_layers + std::max(0, (int)n_layers));
  if (int e = run_relocation(spans, kbufs, seq->d_pos, p, static_cast<hipStream_t>(stream))) return e;
  commit_intervals(seq, runs);
  seq->next_pos = last;
  return ok();
}

static size_t probe_ws(const tu_attn_params* p, int64_t len, int32_t n_probe, int64_t* ld) {
  *ld = (len + kProbeKeys - 1) / kProbeKeys * kProbeKeys;
  const int64_t rows = (int64_t)p->n_q_heads * n_probe;
  return align_up(sizeof(bf16_t) * rows * p->head_dim) + align_up(sizeof(float) * 2 * rows) +
         align_up(sizeof(float) * 2 * rows * (*ld / 32)) + align_up(sizeof(float) * p->n_kv_heads * *ld);
}

size_t attention_probe_workspace_size(const tu_attn_params* p, int64_t len, int32_t n_probe) {
  if (check_attn(p) || len < 0 || n_probe < 0) return 0;
  int64_t ld = 0;
  return std::max<size_t>(probe_ws(p, len, n_probe, &ld), kAlign);
}

int attention_probe(const tu_seq* seq, const void* k_cache, const tu_attn_params* p, const void* q, int32_t n_probe,
                    float weight, float* probs, void* workspace, size_t workspace_bytes, void* stream) {
  if (int e = check_seq(seq)) return e;
  if (int e = check_attn(p)) return e;
  const int G = p->n_q_heads / p->n_kv_heads;
  if (n_probe < 1 || n_probe > seq->len) return fail(TU_ERR_ARG, "n_probe must be in [1, len]");
  if ((int64_t)n_probe * G > kProbeMaxRows)
    return fail(TU_ERR_ARG, "n_probe x query heads per KV head must be at most %d", kProbeMaxRows);
  if ((int64_t)n_probe * p->n_q_heads > 4096) return fail(TU_ERR_ARG, "too many probe rows");
  if (seq->len > INT32_MAX / 2) return fail(TU_ERR_ARG, "context too long");
  if (!std::isfinite(weight)) return fail(TU_ERR_ARG, "weight must be finite");
  if (!k_cache || !q || !probs) return fail(TU_ERR_ARG, "null tensor");
  if (!aligned16(k_cache) || !aligned16(q)) return fail(TU_ERR_ARG, "tensors must be 16-byte aligned");
  int64_t ld = 0;
  const size_t need = probe_ws(p, seq->len, n_probe, &ld);
  if (!workspace || workspace_bytes < need)
    return fail(TU_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
  if (!aligned16(workspace)) return fail(TU_ERR_WORKSPACE, "workspace must be 16-byte aligned");
  Arena ar(workspace);
  const int64_t rows = (int64_t)p->n_q_heads * n_probe;
  ProbeArgs a{};
  a.q = static_cast<const bf16_t*>(q);
  a.q_hat = static_cast<bf16_t*>(ar.take(sizeof(bf16_t) * rows * p->head_dim));
  a.stats = static_cast<float*>(ar.take(sizeof(float) * 2 * rows));
  a.part = static_cast<float*>(ar.take(sizeof(float) * 2 * rows * (ld / 32)));
  a.key_sum = static_cast<float*>(ar.take(sizeof(float) * p->n_kv_heads * ld));
  a.n_parts = (int32_t)(ld / 32);
  a.k_cache = static_cast<const bf16_t*>(k_cache);
  a.pos = seq->d_pos;
  a.probs = probs;
  a.len = (int32_t)seq->len;
  a.n_probe = n_probe;
  a.ld = (int32_t)ld;
  a.n_q_heads = p->n_q_heads;
  a.n_kv_heads = p->n_kv_heads;
  a.head_dim = p->head_dim;
  a.rotary_dim = p->rotary_dim;
  a.theta = p->rope_theta;
  a.scale = p->softmax_scale;
  a.weight = weight;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (int e = hip_check(timed("probe", st, [&] { return launch_probe(a, st); }), "probe launch")) return e;
  return ok();
}

static int group_blocks(int64_t len) {
  return (int)std::min<int64_t>(kGroupMaxBlocks, std::max<int64_t>(1, (len + kGroupMinRows - 1) / kGroupMinRows));
}

size_t attention_group_mass_workspace_size(int64_t len, int32_t n_groups) {
  if (len < 0) return 0;
  return align_up(sizeof(double) * 2 * (size_t)group_blocks(len) * (size_t)std::max(1, (int)n_groups));
}

int attention_group_mass(const tu_seq* seq, const float* probs, const int64_t* groups, int32_t n_groups,
                         int32_t window, float* mass, float* window_mass, float* summary, void* workspace,
                         size_t workspace_bytes, void* stream) {
  if (int e = check_seq(seq)) return e;
  if (n_groups < 1 || n_groups > (1 << 20) || !groups) return fail(TU_ERR_ARG, "1 .. 2^20 groups");
  if (window < 0) return fail(TU_ERR_ARG, "negative window");
  if (!probs || !mass) return fail(TU_ERR_ARG, "null tensor");
  int64_t prev = INT64_MIN;
  for (int g = 0; g < n_groups; ++g) {
    const int64_t a = groups[2 * g], b = groups[2 * g + 1];
    if (b <= a || a < prev || a < 0 || b > INT32_MAX)
      return fail(TU_ERR_RANGE, "group %d [%lld,%lld): groups must be non-empty, sorted, disjoint, in [0, 2^31 - 1)", g,
                  (long long)a, (long long)b);
    prev = b;
  }
  if (seq->len > INT32_MAX / 2) return fail(TU_ERR_ARG, "context too long");
  const size_t need = attention_group_mass_workspace_size(seq->len, n_groups);
  if (!workspace || workspace_bytes < need)
    return fail(TU_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
  if (!aligned16(workspace)) return fail(TU_ERR_WORKSPACE, "workspace must be 16-byte aligned");
  hipStream_t st = static_cast<hipStream_t>(stream);
  GroupArgs a{};
  a.pos = seq->d_pos;
  a.probs = probs;
  a.partial = static_cast<double*>(workspace);
  a.mass = mass;
  a.window_mass = window_mass;
  a.summary = summary;
  a.len = (int32_t)seq->len;
  a.n_total = n_groups;
  a.window = window;
  a.n_blocks = group_blocks(seq->len);
  a.block_rows = (int32_t)(((seq->len + a.n_blocks - 1) / a.n_blocks + 255) / 256 * 256);
  for (int g0 = 0; g0 < n_groups; g0 += kMaxGroupsPerLaunch) {
    a.g_begin = g0;
    a.n = std::min(kMaxGroupsPerLaunch, n_groups - g0);
    for (int g = 0; g < a.n; ++g) {
      a.range[g][0] = (int32_t)groups[2 * (g0 + g)];
      a.range[g][1] = (int32_t)groups[2 * (g0 + g) + 1];
    }
    if (int e = hip_check(timed("group_mass", st, [&] { return launch_group_mass(a, st); }), "group mass")) return e;
  }
  if (int e = hip_check(timed("group_mass", st, [&] { return launch_group_final(a, st); }), "group summary")) return e;
  return ok();
}

size_t attention_tv_workspace_size(int64_t n) {
  if (n < 0) return 0;
  return align_up(sizeof(double) * (size_t)std::max<int64_t>(1, (n + kTvRowsPerBlock - 1) / kTvRowsPerBlock));
}

int attention_tv_distance(const float* p, const float* q, const int32_t* q_row_of_p, int64_t n, float* tv,
                          void* workspace, size_t workspace_bytes, void* stream) {
  if (n < 0 || n > INT32_MAX) return fail(TU_ERR_ARG, "n outside [0, 2^31 - 1]");
  if ((n > 0 && (!p || !q)) || !tv) return fail(TU_ERR_ARG, "null tensor");
  const size_t need = attention_tv_workspace_size(n);
  if (!workspace || workspace_bytes < need)
    return fail(TU_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
  if (!aligned16(workspace)) return fail(TU_ERR_WORKSPACE, "workspace must be 16-byte aligned");
  TvArgs a{};
  a.p = p;
  a.q = q;
  a.map = q_row_of_p;
  a.partial = static_cast<double*>(workspace);
  a.tv = tv;
  a.n = n;
  a.n_blocks = (int32_t)((n + kTvRowsPerBlock - 1) / kTvRowsPerBlock);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (int e = hip_check(timed("tv_distance", st, [&] { return launch_tv(a, st); }), "tv launch")) return e;
  return ok();
}

int tu_profile_enable(int on) {
  g_prof = on != 0;
  return ok();
}

int tu_profile_collect(char* names, int32_t name_stride, int32_t* counts, double* total_ms, int32_t max_entries) {
  if (max_entries < 0 || (max_entries > 0 && (!names || !counts || !total_ms || name_stride < 2)))
    return fail(TU_ERR_ARG, "bad output arrays");
  std::vector<std::string> keys;
  std::vector<int32_t> cnt;
  std::vector<double> sum;
  int status = TU_OK;
  for (auto& r : g_recs) {
    float ms = 0.f;
    if (hipEventSynchronize(r.stop) != hipSuccess || hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess)
      status = fail(TU_ERR_HIP, "event timing failed");
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
    size_t k = 0;
    while (k < keys.size() && keys[k] != r.name) ++k;
    if (k == keys.size()) {
      keys.push_back(r.name);
      cnt.push_back(0);
      sum.push_back(0.0);
    }
    cnt[k] += 1;
    sum[k] += ms;
  }
  g_recs.clear();
  if (status != TU_OK) return status;
  const int n = std::min<int>((int)keys.size(), max_entries);
  for (int i = 0; i < n; ++i) {
    snprintf(names + (size_t)i * name_stride, name_stride, "%s", keys[i].c_str());
    counts[i] = cnt[i];
    total_ms[i] = sum[i];
  }
  ok();
  return n;
}

int tu_validate_update(const tu_update* u) {
  StackPlan sp;
  if (int e = validate_stack(u, &sp)) return e;
  return ok();
}

int update_layer_stack(const tu_update* u, void* workspace, size_t workspace_bytes, void* stream) {
  StackPlan sp;
  if (int e = validate_stack(u, &sp)) return e;
  const StackWorkspace ws = stack_workspace(u, sp);
  const size_t need = ws.total();
  if (!workspace || workspace_bytes < need)
    return fail(TU_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes, need);
  if (!aligned16(workspace)) return fail(TU_ERR_WORKSPACE, "workspace must be 16-byte aligned");
  for (int l = 0; l < u->n_layers; ++l)
    if (u->layers[l].kind == TU_LAYER_ATTN && u->layers[l].vt_cache)
      for (int s = 0; s < u->n_seq; ++s) {
        void* vt = u->layers[l].vt_cache[s];
        if (vt && !aligned16(vt)) return fail(TU_ERR_ARG, "layer %d context %d: V^T copy must be 16-byte aligned", l, s);
      }
  hipStream_t st = static_cast<hipStream_t>(stream);
  const CallStatus status = call_status(workspace);
  void* ws_attn = after_status(workspace);
  void* ws_delta = static_cast<char*>(ws_attn) + align_up(ws.attn);
  // the call's number is recorded by the first workgroup of each of its launches (a call
  // with nothing to launch records it with a one-workgroup kernel, at the end)
  const uint64_t launches = g_launches;

  // Delta layers depend on nothing the attention path writes (the layers' inputs are
  // given), so they run on a side stream of this device, forked after the work
  // already queued on `st` and joined back before returning: every result is then
  // ordered on `st` as if the layers had run in sequence.
  int n_delta = 0;
  for (int l = 0; l < u->n_layers; ++l) n_delta += u->layers[l].kind == TU_LAYER_DELTA;
  SideStream* side = nullptr;
  if (n_delta > 0 && (sp.n_attn > 0 || n_delta < u->n_layers)) {
    if (int e = side_stream(&side)) return e;
    if (int e = hip_check(hipEventRecord(side->fork, st), "fork event")) return e;
    if (int e = hip_check(hipStreamWaitEvent(side->stream, side->fork, 0), "side stream wait")) return e;
  }
  hipStream_t sd = side ? side->stream : st;
  // Everything from here on is enqueued after the fork; a failing launch still joins
  // the side stream back into `st` before the error is returned.
  const int status_code = [&]() -> int {
    if (n_delta > 0) {
      size_t b = 0;
      auto items = stack_delta_items(u, sp);
      std::vector<DeltaArgs> ls;
      plan_delta(&u->delta, items, ws_delta, status, &ls, &b);
      if (int e = run_delta(ls, &u->delta, sd)) return e;
      if (side)
        if (int e = hip_check(hipEventRecord(side->join, side->stream), "join event")) return e;
    }
    // a2-a3: keep-scan and in-place row move over every attention layer of every context
    if (sp.n_attn) {
      auto items = stack_compact_items(u, sp);
      CompactPlan cp;
      if (int e = plan_compaction(items, u->attn.n_kv_heads * u->attn.head_dim * 2, ws_attn, status, &cp)) return e;
      if (int e = run_compaction(cp, st)) return e;
    }
    // a4-a5: the attention layers are independent of each other once the caches are
    // compacted; the layers too small to fill the chip share one set of launches. An
    // attention workgroup holds a whole CU, and so does a delta-chain workgroup: an
    // attention launch of kGateWaves or more full waves leaves no CU idle for the delta
    // layers to use, so it waits for them (they run beside the compaction and the
    // stage) instead of sharing CUs with them, which would only lengthen it by as much.
    // Shorter launches leave CUs idle at their ragged end and keep the overlap.
    hipEvent_t gate = side ? side->join : nullptr;
    for (auto& items : stack_attn_groups(u, sp)) {
      size_t b = 0;
      std::vector<AttnLaunch> ls;
      plan_attention(&u->attn, items, ws_attn, status, &ls, &b);
      int64_t wgs = 0;
      for (const auto& L : ls) wgs += L.order.blocks > 0 ? L.order.blocks : L.attn.total_items;
      const bool wait = gate && wgs >= (int64_t)kGateWaves * kCus;
      if (int e = run_attention(ls, u->attn.head_dim, st, wait ? gate : nullptr)) return e;
      if (wait) gate = nullptr;
    }
    // tail-and-relocate: the stored keys of the tail turn from their computed
    // positions to the placed ones (values and recurrent state stay as computed)
    for (int s = 0; s < u->n_seq && sp.n_attn; ++s) {
      const tu_seq_update& su = u->seqs[s];
      if (su.placement != TU_PLACE_RELOCATE || su.T == 0) continue;
      const int64_t L_keep = su.seq->len - sp.rc[s].removed;
      std::vector<RelocSpan> spans;
      for (int q = 0, t0 = 0; q < su.n_place_runs; ++q) {
        const int64_t n = su.place_runs[2 * q + 1] - su.place_runs[2 * q];
        const int64_t delta = su.place_runs[2 * q] - (su.seq->next_pos + t0);
        if (delta != 0) spans.push_back({L_keep + t0, n, delta});
        t0 += (int)n;
      }
      std::vector<void*> kbufs;
      for (int l = 0; l < u->n_layers; ++l)
        if (u->layers[l].kind == TU_LAYER_ATTN) kbufs.push_back(u->layers[l].k_cache[s]);
      if (int e = run_relocation(spans, kbufs, su.seq->d_pos, &u->attn, st)) return e;
    }
    // rows of the tail removed once it is prefilled (maintenance delimiters): their
    // direct KV goes, their effect on the recurrent state and on later rows stays
    if (sp.n_attn && sp.any_post) {
      auto items = stack_post_items(u, sp);
      CompactPlan cp;
      if (int e = plan_compaction(items, u->attn.n_kv_heads * u->attn.head_dim * 2, ws_attn, status, &cp)) return e;
      if (int e = run_compaction(cp, st)) return e;
    }
    return TU_OK;
  }();
  if (side) {
    const std::string err = g_err;   // the join must not hide the launch error
    int e = hip_check(hipEventRecord(side->join, side->stream), "join event");
    if (!e) e = hip_check(hipStreamWaitEvent(st, side->join, 0), "join wait");
    if (status_code != TU_OK) {
      g_err = err;
      return status_code;
    }
    if (e) return e;
  }
  if (status_code != TU_OK) return status_code;
  if (g_launches == launches)
    if (int e = hip_check(launch_status_mark(status, st), "status mark")) return e;
  // a8: commit metadata
  for (int s = 0; s < u->n_seq; ++s) {
    tu_seq* seq = u->seqs[s].seq;
    const bool post = sp.n_attn && sp.post_rc[s].removed > 0;
    const int64_t L_keep = seq->len - sp.rc[s].removed;
    commit_intervals(seq, post ? sp.post_rc[s].live_after : sp.final_iv[s]);
    seq->len = L_keep + u->seqs[s].T - (post ? sp.post_rc[s].removed : 0);
    seq->next_pos = sp.cursor_after[s];
    // the V^T copies now hold every row up to the tail's end, except rows the removal
    // after the prefill moved
    if (sp.n_attn) seq->vt_rows = post ? sp.post_rc[s].first_row : seq->len;
    else seq->vt_rows = std::min(seq->vt_rows, sp.rc[s].removed > 0 ? sp.rc[s].first_row : seq->len);
  }
  return ok();
}

}  // extern "C"
