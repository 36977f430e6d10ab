// C-ABI entry points: argument checks, the k:(F-k) mask builder, compaction of
// the frame mask into a kept-tile list and a work plan (query frames with many
// kept frames split into balanced pieces), a bounded cache of the device copies of
// those plans, a
// per-(device, stream) workspace for the partial results of split frames, and
// dispatch of the gfx950 kernels on the caller's stream.
#include "../../include/tile_attn.h"

#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cfloat>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <map>
#include <mutex>
#include <numeric>
#include <string>
#include <utility>
#include <vector>

#include "launch.h"
#include "host_internal.h"
#include "plan_cache.h"

namespace ta {
namespace host {

thread_local std::string g_last_error;

int fail(int status, const std::string& detail) {
  g_last_error = detail;
  return status;
}

void clear_error() { g_last_error.clear(); }

void compact_host(const uint8_t* mask, int F, int32_t* row_ptr, uint16_t* cols,
                  uint16_t* order, int* nnz_out) {
  int nnz = 0;
  row_ptr[0] = 0;
  for (int i = 0; i < F; ++i) {
    for (int j = 0; j < F; ++j)
      if (mask[(size_t)i * F + j]) cols[nnz++] = (uint16_t)j;
    row_ptr[i + 1] = nnz;
  }
  if (order) {
    std::vector<int> idx(F);
    std::iota(idx.begin(), idx.end(), 0);
    std::stable_sort(idx.begin(), idx.end(), [&](int a, int b) {
      return row_ptr[a + 1] - row_ptr[a] > row_ptr[b + 1] - row_ptr[b];
    });
    for (int i = 0; i < F; ++i) order[i] = (uint16_t)idx[i];
  }
  *nnz_out = nnz;
}

// Work plan of one mask. Every query frame is one work item over its kept key
// frames, except that a frame keeping more than twice the mean number of kept
// frames per row (rounded up) is split into items of about that mean size: those
// items write partial results (slot >= 0) that a merge pass combines. Splitting
// keeps one heavy row (the global query frames of the symmetric mask keep every
// frame) from setting the critical path while the other workgroups idle.
struct WorkPlan {
  std::vector<int32_t> items;  // 4 per item: frame, first kept entry, count, slot
  std::vector<int32_t> cols;   // kept key frames, row after row
  std::vector<int32_t> heavy;  // 3 per split frame: frame, first slot, slots
  int n_slots = 0;
};

constexpr int kMaxChunksPerFrame = 32;

WorkPlan plan_work(const uint8_t* mask, int F, bool allow_split) {
  WorkPlan pl;
  std::vector<int32_t> row_ptr(F + 1);
  std::vector<uint16_t> cols((size_t)F * F + 1), order(F);
  int nnz = 0;
  compact_host(mask, F, row_ptr.data(), cols.data(), order.data(), &nnz);
  pl.cols.assign(cols.begin(), cols.begin() + nnz);
  if (pl.cols.empty()) pl.cols.push_back(0);
  const int chunk = std::max(1, (nnz + F - 1) / F);  // mean kept frames per row, rounded up
  struct Item { int frame, beg, cnt, slot; };
  std::vector<Item> list;
  for (int i = 0; i < F; ++i) {
    const int beg = row_ptr[i], cnt = row_ptr[i + 1] - row_ptr[i];
    int pieces = 1;
    if (allow_split && cnt > 2 * chunk) pieces = std::min((cnt + chunk - 1) / chunk, kMaxChunksPerFrame);
    if (pieces == 1) {
      list.push_back({i, beg, cnt, -1});
      continue;
    }
    pl.heavy.insert(pl.heavy.end(), {i, pl.n_slots, pieces});
    for (int p = 0; p < pieces; ++p) {
      const int b0 = beg + (int)((int64_t)cnt * p / pieces);
      const int b1 = beg + (int)((int64_t)cnt * (p + 1) / pieces);
      list.push_back({i, b0, b1 - b0, pl.n_slots++});
    }
  }
  // Longest items first; ties keep frame and piece order.
  std::stable_sort(list.begin(), list.end(),
                   [](const Item& x, const Item& y) { return x.cnt > y.cnt; });
  for (const Item& it : list) pl.items.insert(pl.items.end(), {it.frame, it.beg, it.cnt, it.slot});
  return pl;
}

HostWorkList build_work_list(const uint8_t* masks, int n_masks, int H, int F, bool allow_split) {
  std::vector<int32_t> items, cols, heavy;
  int n_slots = 0;
  WorkPlan shared;
  if (n_masks == 1) {
    shared = plan_work(masks, F, allow_split);
    cols = shared.cols;
  }
  for (int h = 0; h < H; ++h) {
    WorkPlan own;
    if (n_masks != 1) own = plan_work(masks + (size_t)h * F * F, F, allow_split);
    const WorkPlan& pl = n_masks == 1 ? shared : own;
    const int col_off = n_masks == 1 ? 0 : (int)cols.size();
    if (n_masks != 1) cols.insert(cols.end(), pl.cols.begin(), pl.cols.end());
    for (size_t i = 0; i < pl.items.size(); i += 4) {
      const int slot = pl.items[i + 3];
      items.insert(items.end(), {h, pl.items[i], pl.items[i + 1] + col_off, pl.items[i + 2],
                                 slot < 0 ? -1 : slot + n_slots});
    }
    for (size_t i = 0; i < pl.heavy.size(); i += 3)
      heavy.insert(heavy.end(), {h, pl.heavy[i], pl.heavy[i + 1] + n_slots, pl.heavy[i + 2]});
    n_slots += pl.n_slots;
  }
  HostWorkList hw;
  hw.words.insert(hw.words.end(), items.begin(), items.end());
  hw.off_cols = hw.words.size();
  hw.words.insert(hw.words.end(), cols.begin(), cols.end());
  hw.off_heavy = hw.words.size();
  hw.words.insert(hw.words.end(), heavy.begin(), heavy.end());
  if (heavy.empty()) hw.words.push_back(0);
  hw.n_items = (int)(items.size() / 5);
  hw.n_heavy = (int)(heavy.size() / 4);
  hw.n_slots = n_slots;
  return hw;
}

DeviceWorkList place_work_list(const HostWorkList& hw, void* buf) {
  DeviceWorkList wl;
  const int32_t* w = static_cast<const int32_t*>(buf);
  wl.buffer = buf;
  wl.items = w;
  wl.cols = w + hw.off_cols;
  wl.heavy = w + hw.off_heavy;
  wl.n_items = hw.n_items;
  wl.n_heavy = hw.n_heavy;
  wl.n_slots = hw.n_slots;
  if (hw.wg_per_xcd > 0) {
    wl.sched_xcd = w + hw.off_xcd;
    wl.cut_units = w + hw.off_cut_units;
    wl.n_cut_units = hw.n_cut_units;
    wl.n_part_slots = hw.n_part_slots;
    wl.wg_per_xcd = hw.wg_per_xcd;
    wl.unit_table = hw.unit_table;
  }
  return wl;
}

void append_fwd_schedule(HostWorkList& hw, int B, int nqb, int rows, int d, int T, int P, int F,
                         int slots_x, bool share_tail, bool by_length) {
  const int32_t* items = hw.words.data();
  const int32_t* cols = hw.words.data() + hw.off_cols;
  const int64_t n_items = hw.n_items;
  const int tpf = (T + 63) / 64, ptiles = (P + 63) / 64;
  // Kept tiles of item i for one query block (0 for a query block past its segment).
  auto tiles_of = [&](int64_t i, int qb) -> int64_t {
    const int32_t* it = items + 5 * i;
    const int frame = it[1], beg = it[2], cnt = it[3];
    const int seg_len = (P > 0 && frame == F) ? P : T;
    if ((int64_t)qb * rows >= seg_len) return 0;
    int64_t t = (int64_t)cnt * tpf;
    if (P > 0 && cnt > 0 && cols[beg + cnt - 1] == F) t += ptiles - tpf;
    return t;
  };
  const int64_t per_b = n_items * nqb, n = (int64_t)B * per_b;
  auto unit_tiles = [&](int64_t u) { return tiles_of((u % per_b) / nqb, (int)(u % nqb)); };
  // A query block past its segment's end (the text segment is shorter than the blocks
  // the video needs) has no rows: nothing to run.
  auto has_rows = [&](int64_t u) {
    const int32_t* it = items + 5 * ((u % per_b) / nqb);
    const int seg_len = (P > 0 && it[1] == F) ? P : T;
    return (int64_t)(u % nqb) * rows < seg_len;
  };
  // Where every segment ends on a query block of at most 32 rows (video only, d = 64
  // or 96), the kernel runs those blocks on two waves, after the full blocks of each
  // XCD's share, and they already even out the last round: no parts then.
  const bool short_last = P == 0 && (d == 64 || d == 96) && nqb > 1 && T - (nqb - 1) * rows <= 32;
  std::vector<int32_t> xcd(4 * 8), pieces, cut_units;
  int n_part_slots = 0;
  int64_t wg_max = 0;
  // Longest first where it changes something: a plan with split frames runs the
  // kernel's persistent loop instead (its queue takes the natural order), and a share
  // whose units with rows already come longest first keeps the contiguous form.
  const int64_t q = n / 8, r = n % 8;
  bool table = false;
  if (by_length && hw.n_heavy == 0) {
    for (int x = 0; x < 8 && !table; ++x) {
      const int64_t start = x * q + std::min<int64_t>(x, r), cnt = q + (x < r);
      int64_t prev = -1;
      for (int64_t u = start; u < start + cnt && !table; ++u) {
        if (!has_rows(u)) continue;
        const int64_t len = unit_tiles(u);
        table = prev >= 0 && len > prev;
        prev = len;
      }
    }
  }
  std::vector<int64_t> us;
  for (int x = 0; x < 8; ++x) {
    const int64_t start = x * q + std::min<int64_t>(x, r), cnt = q + (x < r);
    int64_t n_dp = cnt;
    const int64_t first_piece = (int64_t)pieces.size() / 4;
    // This XCD's units in the order it runs them: as numbered, or longest first.
    us.resize(cnt);
    for (int64_t i = 0; i < cnt; ++i) us[i] = start + i;
    if (table)
      std::stable_sort(us.begin(), us.end(),
                       [&](int64_t a, int64_t b) { return unit_tiles(a) > unit_tiles(b); });
    // An XCD runs its whole units in rounds of slots_x. If the last round is ragged,
    // its R units can be cut into k parts each: the parts then take ceil(R k / slots_x)
    // rounds of 1/k of a unit instead of one round of whole units, and every part
    // writes its rows' O/l and log-sum-exp (fp32) for a merge pass to read back. The k
    // of the largest net saving is taken: the time saved (a tile of 64 keys for one
    // workgroup's query rows takes about 2.8 us at d = 96 and 256 rows, in proportion
    // to d and the rows) less the partial traffic of all XCDs at about 4 TB/s. A plan
    // with split frames is left whole: its pieces, dispatched longest first, already
    // even out the last round, and parts of pieces would add a second merge.
    const int64_t ragged = cnt % slots_x;
    int parts_k = 1;
    if (share_tail && hw.n_heavy == 0 && !short_last && cnt > slots_x && ragged > 0) {
      double mean_tiles = 0;
      for (int64_t i = cnt - ragged; i < cnt; ++i) mean_tiles += (double)unit_tiles(us[i]);
      mean_tiles /= (double)ragged;
      const double tile_s = 2.8e-6 * (rows / 256.0) * (d / 96.0);
      const double part_s = 8.0 * rows * (d + 4) * 4.0 * 2.0 / 4.0e12;  // per part, all XCDs
      int best_k = 1;
      double best = 0.0;
      for (int kk = 2; kk <= 16; ++kk) {
        const double rounds = (double)((ragged * kk + slots_x - 1) / slots_x) / kk;
        const double net = (1.0 - rounds) * mean_tiles * tile_s - (double)(ragged * kk) * part_s;
        if (net > best) {
          best = net;
          best_k = kk;
        }
      }
      if (best_k > 1 && best > 10e-6) {
        n_dp = cnt - ragged;
        parts_k = best_k;
      }
    }
    if (table) {  // the whole units as table entries, ahead of any parts
      for (int64_t i = 0; i < n_dp; ++i)
        if (has_rows(us[i])) pieces.insert(pieces.end(), {(int32_t)us[i], 0, (int32_t)unit_tiles(us[i]), -1});
    }
    for (int64_t i = n_dp; i < cnt; ++i) {  // the ragged round, in parts
      const int64_t u = us[i];
      const int64_t len = unit_tiles(u);
      const int parts = (int)std::min<int64_t>(parts_k, len);
      if (parts <= 1) {  // a unit of one tile, or of none (its rows still get written), runs whole
        if (has_rows(u)) pieces.insert(pieces.end(), {(int32_t)u, 0, (int32_t)len, -1});
        continue;
      }
      cut_units.insert(cut_units.end(), {(int32_t)u, n_part_slots, parts});
      for (int p = 0; p < parts; ++p) {
        const int64_t t0 = len * p / parts, t1 = len * (p + 1) / parts;
        pieces.insert(pieces.end(), {(int32_t)u, (int32_t)t0, (int32_t)(t1 - t0), n_part_slots++});
      }
    }
    if (table) n_dp = 0;  // every position is a table entry
    const int64_t n_part = (int64_t)pieces.size() / 4 - first_piece;
    xcd[4 * x] = (int32_t)start;
    xcd[4 * x + 1] = (int32_t)n_dp;
    xcd[4 * x + 2] = (int32_t)n_part;
    xcd[4 * x + 3] = (int32_t)first_piece;
    wg_max = std::max(wg_max, n_dp + n_part);
  }
  hw.n_cut_units = (int)(cut_units.size() / 3);
  if (pieces.empty()) pieces.assign(4, 0);
  if (cut_units.empty()) cut_units.assign(3, 0);
  hw.off_xcd = hw.words.size();
  hw.words.insert(hw.words.end(), xcd.begin(), xcd.end());
  hw.off_pieces = hw.words.size();
  hw.words.insert(hw.words.end(), pieces.begin(), pieces.end());
  hw.off_cut_units = hw.words.size();
  hw.words.insert(hw.words.end(), cut_units.begin(), cut_units.end());
  hw.n_part_slots = n_part_slots;
  hw.wg_per_xcd = (int)wg_max;
  hw.unit_table = table;
}

// A cached plan: its device buffer and, per stream that enqueued work with it, an
// event recorded after that work (stream order makes the latest one cover the
// earlier ones on the same stream).
struct CachedPlan {
  DeviceWorkList wl;
  int dev = 0;
  std::vector<std::pair<void*, hipEvent_t>> uses;
};

struct HipPlanOps {
  bool idle(CachedPlan& p) {
    bool done = true;
    for (auto& u : p.uses) done = done && hipEventQuery(u.second) != hipErrorNotReady;
    (void)hipGetLastError();  // a pending event's status is not an error of the caller's
    return done;
  }
  void release(CachedPlan& p) {
    int cur = 0;
    const bool restore = hipGetDevice(&cur) == hipSuccess && cur != p.dev;
    if (restore) (void)hipSetDevice(p.dev);
    (void)hipFree(p.wl.buffer);
    for (auto& u : p.uses) (void)hipEventDestroy(u.second);
    if (restore) (void)hipSetDevice(cur);
    (void)hipGetLastError();
  }
};

std::mutex g_cache_mutex;
ta::PlanCache<CachedPlan, HipPlanOps> g_cache(TA_PLAN_CACHE_ENTRIES);

// A plan acquired for one call: a copy of its device addresses, and the cache slot the
// call holds until end_plan_use() (so no eviction frees it before the call's kernels are
// enqueued and their completion can be tracked).
struct PlanUse {
  DeviceWorkList wl;
  ta::PlanCache<CachedPlan, HipPlanOps>::Handle slot = nullptr;
};

// Returns the device-resident work list for H heads with n_masks masks (1: shared,
// H: one per head), split or not, uploading it on first use on device dev.
// The forward launch a plan is scheduled for (append_fwd_schedule).
struct FwdLaunch {
  int B, nqb, rows, d, T, P, F, slots_x;
  bool share_tail, by_length;
};

int work_list_for(const uint8_t* masks, int n_masks, int H, int F, bool allow_split, int dev,
                  PlanUse* out, const FwdLaunch* fl = nullptr) {
  std::string key(reinterpret_cast<const char*>(masks), (size_t)n_masks * F * F);
  key += allow_split ? "|s|" : "|u|";
  key += std::to_string(H) + "|" + std::to_string(n_masks) + "|" + std::to_string(F) + "|" +
         std::to_string(dev);
  if (fl)
    for (int v : {fl->B, fl->nqb, fl->rows, fl->d, fl->T, fl->P, fl->F, fl->slots_x, (int)fl->share_tail,
                  (int)fl->by_length})
      key += "|" + std::to_string(v);
  std::lock_guard<std::mutex> lock(g_cache_mutex);
  if (auto h = g_cache.acquire(key)) {
    out->wl = h->value.wl;
    out->slot = h;
    return TA_OK;
  }
  HostWorkList hw = build_work_list(masks, n_masks, H, F, allow_split);
  if (fl)
    append_fwd_schedule(hw, fl->B, fl->nqb, fl->rows, fl->d, fl->T, fl->P, fl->F, fl->slots_x,
                        fl->share_tail, fl->by_length);
  const size_t total = hw.words.size() * sizeof(int32_t);
  void* buf = nullptr;
  hipError_t e = hipMalloc(&buf, total);
  if (e != hipSuccess) return fail(TA_ERR_HIP, std::string("hipMalloc: ") + hipGetErrorString(e));
  e = hipMemcpy(buf, hw.words.data(), total, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(buf);
    return fail(TA_ERR_HIP, std::string("hipMemcpy: ") + hipGetErrorString(e));
  }
  CachedPlan cp;
  cp.wl = place_work_list(hw, buf);
  cp.dev = dev;
  auto h = g_cache.insert(std::move(key), std::move(cp));
  out->wl = h->value.wl;
  out->slot = h;
  return TA_OK;
}

// The call has enqueued every kernel that reads the plan on `stream` (or failed to):
// record an event after them, or, when the stream is being captured into a graph that
// may replay at any later time, keep the plan for the rest of the process.
void end_plan_use(PlanUse& u, void* stream) {
  if (!u.slot) return;
  std::lock_guard<std::mutex> lock(g_cache_mutex);
  const hipStream_t s = static_cast<hipStream_t>(stream);
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) {
    (void)hipGetLastError();
    g_cache.pin(u.slot);
  } else {
    auto& uses = u.slot->value.uses;
    auto it = std::find_if(uses.begin(), uses.end(),
                           [&](const std::pair<void*, hipEvent_t>& x) { return x.first == stream; });
    hipEvent_t ev = nullptr;
    if (it != uses.end()) {
      ev = it->second;
    } else if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) == hipSuccess) {
      uses.emplace_back(stream, ev);
    } else {
      ev = nullptr;
    }
    if (!ev || hipEventRecord(ev, s) != hipSuccess) {
      (void)hipGetLastError();
      g_cache.pin(u.slot);  // completion cannot be tracked: never free it
    }
  }
  g_cache.release(u.slot);
  u.slot = nullptr;
}

// Holds a plan for the duration of a call and ends its use on every return path.
struct PlanGuard {
  PlanUse use;
  void* stream;
  explicit PlanGuard(void* s) : stream(s) {}
  ~PlanGuard() { end_plan_use(use, stream); }
};

int resident_slots_per_xcd(int dev) {
  static std::mutex mu;
  static std::map<int, int> slots;
  std::lock_guard<std::mutex> lock(mu);
  auto it = slots.find(dev);
  if (it == slots.end()) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 8) {
      (void)hipGetLastError();
      cus = 256;  // MI355X
    }
    it = slots.emplace(dev, 2 * (cus / 8)).first;  // two forward workgroups per compute unit
  }
  return it->second;
}

// Partial-result workspace of split frames, one per (device, stream) so that calls
// on different streams never share it; replaced by a larger one on demand, every
// buffer kept until process exit.
struct Workspace {
  void* ptr = nullptr;
  size_t bytes = 0;
  std::vector<void*> retired;
  int* queue = nullptr;  // the forward kernel's work-queue counters, never replaced
};
std::map<std::pair<int, void*>, Workspace> g_workspaces;

// Largest workspace a call may use; masks that would need more are not split.
constexpr size_t kMaxWorkspaceBytes = size_t(2) << 30;

bool ranges_overlap(const void* a, size_t na, const void* b, size_t nb) {
  auto x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

int check_args(const void* q, const void* k, const void* v, void* out, int B, int H, int F,
               int T, int d, float scale, int P) {
  if (!q || !k || !v || !out) return fail(TA_ERR_NULL_PTR, "q, k, v and out must be non-NULL");
  if (B < 1 || H < 1 || F < 1 || T < 1)
    return fail(TA_ERR_BAD_SHAPE, "B, H, F and T must be >= 1");
  if (P < 0) return fail(TA_ERR_BAD_SHAPE, "the text prefix length must be >= 0");
  if (F > TA_MAX_FRAMES) return fail(TA_ERR_BAD_SHAPE, "F exceeds TA_MAX_FRAMES");
  if ((int64_t)F * T + P > INT32_MAX) return fail(TA_ERR_BAD_SHAPE, "P + F * T exceeds 2^31 - 1");
  if (d != 64 && d != 96 && d != 128) return fail(TA_ERR_HEAD_DIM, "d must be 64, 96 or 128");
  const int rows = ta::fwd_rows_per_workgroup(d) > 0 ? ta::fwd_rows_per_workgroup(d) : 256;
  const int64_t nqb = (std::max(T, P) + rows - 1) / rows;
  const int64_t n_wg = (int64_t)B * H * (F + (P > 0)) * nqb;
  if (n_wg * ta::kThreads > (int64_t)UINT32_MAX)
    return fail(TA_ERR_BAD_SHAPE, "B * H * F * ceil(T / 256) workgroups exceed the grid limit");
  if (!std::isfinite(scale)) return fail(TA_ERR_BAD_SCALE, "scale must be finite");
  for (const void* p : {q, k, v, (const void*)out})
    if (reinterpret_cast<uintptr_t>(p) % 16)
      return fail(TA_ERR_ALIGN, "q, k, v and out must be 16-byte aligned");
  const size_t bytes = (size_t)B * H * ((size_t)F * T + P) * d * 2;
  for (const void* p : {q, k, v})
    if (ranges_overlap(out, bytes, p, bytes)) return fail(TA_ERR_OVERLAP, "out overlaps an input");
  return TA_OK;
}


int queue_for(int dev, void* stream, int** out) {
  std::lock_guard<std::mutex> lock(g_cache_mutex);
  Workspace& ws = g_workspaces[{dev, stream}];
  if (!ws.queue) {
    void* p = nullptr;
    hipError_t e = hipMalloc(&p, 64 * sizeof(int));
    if (e != hipSuccess) return fail(TA_ERR_HIP, std::string("hipMalloc: ") + hipGetErrorString(e));
    e = hipMemset(p, 0, 64 * sizeof(int));
    if (e != hipSuccess) {
      (void)hipFree(p);
      return fail(TA_ERR_HIP, std::string("hipMemset: ") + hipGetErrorString(e));
    }
    ws.queue = static_cast<int*>(p);
  }
  *out = ws.queue;
  return TA_OK;
}

// Workspace of at least `bytes` for (dev, stream). One that is too small is replaced
// by a larger one (at least 1.5 times the old size, so replacements stay few) and
// kept allocated until process exit: work already enqueued with it, or being
// enqueued by another thread that was handed it, never sees it freed, and nothing
// has to wait for the stream.
int workspace_for(int dev, void* stream, size_t bytes, void** out) {
  std::lock_guard<std::mutex> lock(g_cache_mutex);
  Workspace& ws = g_workspaces[{dev, stream}];
  if (ws.bytes < bytes) {
    size_t size = std::max(bytes, ws.bytes + ws.bytes / 2);
    void* p = nullptr;
    hipError_t e = hipMalloc(&p, size);
    if (e != hipSuccess && size > bytes) {
      (void)hipGetLastError();
      size = bytes;  // the geometric size may not fit where the exact one does
      e = hipMalloc(&p, size);
    }
    if (e != hipSuccess) return fail(TA_ERR_HIP, std::string("hipMalloc: ") + hipGetErrorString(e));
    if (ws.ptr) ws.retired.push_back(ws.ptr);
    ws.ptr = p;
    ws.bytes = size;
  }
  *out = ws.ptr;
  return TA_OK;
}

int enqueue_fwd(const void* q, const void* k, const void* v, void* out, int B, int H, int F,
                int T, int d, int P, const DeviceWorkList& plan, float* ws, float scale,
                float* lse, void* stream, int* queue, int slots_x) {
  const DeviceWorkList* wl = &plan;
  const int L = std::max(T, P);
  hipError_t e;
  ta::FwdArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.out = static_cast<uint16_t*>(out);
  a.B = B;
  a.H = H;
  a.F = F;
  a.T = T;
  a.d = d;
  a.P = P;
  a.items = wl->items;
  a.cols = wl->cols;
  a.n_items = wl->n_items;
  // ws: [frame pieces' O/l][their lse][parts of units: O/l and lse per row]
  const size_t frame_rows = (size_t)wl->n_slots * B * L;
  a.ws_o = ws;
  a.ws_lse = ws ? ws + frame_rows * d : nullptr;
  a.ws_parts = ws ? ws + frame_rows * (d + 1) : nullptr;
  a.sched = wl->sched_xcd;
  a.cut_units = wl->cut_units;
  a.n_cut_units = wl->n_cut_units;
  a.wg_per_xcd = wl->wg_per_xcd;
  a.unit_table = wl->unit_table;
  a.slots_per_xcd = std::max(1, slots_x);
  a.queue = queue;
  a.lse = lse;
  // Logits are formed from |scale| (a negative scale flips the sign of q, which
  // is exact in bf16). scale == 0 zeroes q instead, so every logit is exactly 0
  // and the weights exactly uniform; c only has to stay positive.
  if (scale == 0.f) {
    a.c = 1.f;
    a.qflip = 0u;
    a.qmask = 0u;
  } else {
    a.c = std::max(std::fabs(scale) * 1.4426950408889634f, FLT_MIN);
    a.qflip = std::signbit(scale) ? 0x80008000u : 0u;
    a.qmask = 0xFFFFFFFFu;
  }
  if (wl->wg_per_xcd == 0) {  // nothing to run (no query block has rows)
    g_last_error.clear();
    return TA_OK;
  }
  e = ta::launch_tile_attn_fwd(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(TA_ERR_HIP, std::string("kernel launch: ") + hipGetErrorString(e));
  if (wl->n_heavy > 0) {
    ta::MergeArgs m;
    m.ws_o = a.ws_o;
    m.ws_lse = a.ws_lse;
    m.heavy = wl->heavy;
    m.n_heavy = wl->n_heavy;
    m.B = B;
    m.H = H;
    m.F = F;
    m.T = T;
    m.d = d;
    m.P = P;
    m.out = a.out;
    m.lse = lse;
    e = ta::launch_merge_partials(m, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail(TA_ERR_HIP, std::string("merge launch: ") + hipGetErrorString(e));
  }
  return TA_OK;
}

int run_fwd(const void* q, const void* k, const void* v, void* out, int B, int H, int F, int T,
            int d, const uint8_t* masks, int n_masks, float scale, float* lse, void* stream,
            int P = 0) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(TA_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  const int L = std::max(T, P);  // longest segment: rows per query-block grid column
  const int64_t nqb = (L + ta::fwd_rows_per_workgroup(d) - 1) / ta::fwd_rows_per_workgroup(d);
  // With a text prefix, plan F + 1 segments: video row i keeps its mask row plus the
  // text (segment F); the text row keeps everything.
  std::vector<uint8_t> aug;
  int n_seg = F;
  if (P > 0) {
    n_seg = F + 1;
    aug.assign((size_t)n_masks * n_seg * n_seg, 1);
    for (int m = 0; m < n_masks; ++m)
      for (int i = 0; i < F; ++i)
        for (int j = 0; j < F; ++j)
          aug[((size_t)m * n_seg + i) * n_seg + j] = masks[((size_t)m * F + i) * F + j] ? 1 : 0;
    masks = aug.data();
  }
  const int rows = ta::fwd_rows_per_workgroup(d);
  // The MM-DiT form's units differ much in length (text and global rows keep every
  // segment, other rows a few): each XCD runs its share longest first where that
  // changes the order and the plan splits no frame.
  const FwdLaunch fl{B, (int)nqb, rows, d, T, P, F, resident_slots_per_xcd(dev), true, P > 0};
  PlanGuard plan(stream);
  int st = work_list_for(masks, n_masks, H, n_seg, true, dev, &plan.use, &fl);
  if (st != TA_OK) return st;
  const int64_t max_wg = (int64_t)UINT32_MAX / ta::kThreads;
  auto ws_bytes = [&](const DeviceWorkList& w) {
    return ((size_t)w.n_slots * B * L * (d + 1) + (size_t)w.n_part_slots * rows * (d + 4)) * sizeof(float);
  };
  if (ws_bytes(plan.use.wl) > kMaxWorkspaceBytes || (int64_t)8 * plan.use.wl.wg_per_xcd > max_wg) {
    end_plan_use(plan.use, stream);
    const FwdLaunch plain{B, (int)nqb, rows, d, T, P, F, fl.slots_x, false, fl.by_length};
    st = work_list_for(masks, n_masks, H, n_seg, false, dev, &plan.use, &plain);  // the same rows, not split
    if (st != TA_OK) return st;
  }
  const DeviceWorkList* wl = &plan.use.wl;
  void* ws = nullptr;
  if (ws_bytes(*wl) > 0) {
    st = workspace_for(dev, stream, ws_bytes(*wl), &ws);
    if (st != TA_OK) return st;
  }
  // The MM-DiT form at d = 64 with split frames runs the kernel's persistent work loop:
  // its units mix pieces of the text and global rows, short video units and empty text
  // query blocks, and the hardware's in-order dispatch of one workgroup per unit left
  // slots idle (measured at the CogVideoX shape with one global frame). Without split
  // frames, and for the video-only form, one workgroup per unit was as fast or faster.
  int* queue = nullptr;
  if (P > 0 && d == 64 && wl->n_heavy > 0 && (st = queue_for(dev, stream, &queue)) != TA_OK) return st;
  st = enqueue_fwd(q, k, v, out, B, H, F, T, d, P, *wl, static_cast<float*>(ws), scale, lse, stream, queue,
                   fl.slots_x);
  if (st != TA_OK) return st;
  g_last_error.clear();
  return TA_OK;
}


// Gradients: prep (lse in base 2, delta), the query-side pass over the forward's
// work list, the key-side pass over the work list of the transposed masks, and
// the sums of split frames. The workspace holds [lse2][delta] (B*H*F*T floats
// each), then the dq partials and the dk, dv partials.
int run_bwd(const void* q, const void* k, const void* v, const void* out, const void* dout,
            const float* lse, void* dq, void* dk, void* dv, int B, int H, int F, int T, int d,
            const uint8_t* masks, int n_masks, float scale, void* stream, int P = 0) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(TA_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  const int64_t max_wg = (int64_t)UINT32_MAX / ta::kThreads;
  const int L = std::max(T, P);  // longest segment
  const int qpw = ta::bwd_queries_per_workgroup(d);
  const int64_t nqb = (L + qpw - 1) / qpw;
  const int kpw = ta::bwd_keys_per_workgroup(d);
  const int64_t nkb = (L + kpw - 1) / kpw;
  const size_t part_row = (size_t)B * L * d * sizeof(float);

  // Segments: the F frames, plus the text (segment F) with a prefix, whose row and
  // column the (F+1) x (F+1) mask keeps entirely.
  const int n_seg = P > 0 ? F + 1 : F;
  std::vector<uint8_t> aug;
  if (P > 0) {
    aug.assign((size_t)n_masks * n_seg * n_seg, 1);
    for (int m = 0; m < n_masks; ++m)
      for (int i = 0; i < F; ++i)
        for (int j = 0; j < F; ++j)
          aug[((size_t)m * n_seg + i) * n_seg + j] = masks[((size_t)m * F + i) * F + j] ? 1 : 0;
    masks = aug.data();
  }
  PlanGuard plan_q(stream), plan_k(stream);
  int st = work_list_for(masks, n_masks, H, n_seg, true, dev, &plan_q.use);
  if (st != TA_OK) return st;
  if ((size_t)plan_q.use.wl.n_slots * part_row > kMaxWorkspaceBytes ||
      (int64_t)B * plan_q.use.wl.n_items * nqb > max_wg) {
    end_plan_use(plan_q.use, stream);
    st = work_list_for(masks, n_masks, H, n_seg, false, dev, &plan_q.use);
    if (st != TA_OK) return st;
  }
  const DeviceWorkList* wq = &plan_q.use.wl;
  std::vector<uint8_t> mt((size_t)n_masks * n_seg * n_seg);
  for (int m = 0; m < n_masks; ++m)
    for (int i = 0; i < n_seg; ++i)
      for (int j = 0; j < n_seg; ++j)
        mt[((size_t)m * n_seg + i) * n_seg + j] = masks[((size_t)m * n_seg + j) * n_seg + i];
  st = work_list_for(mt.data(), n_masks, H, n_seg, true, dev, &plan_k.use);
  if (st != TA_OK) return st;
  if ((size_t)plan_k.use.wl.n_slots * 2 * part_row > kMaxWorkspaceBytes ||
      (int64_t)B * plan_k.use.wl.n_items * nkb > max_wg) {
    end_plan_use(plan_k.use, stream);
    st = work_list_for(mt.data(), n_masks, H, n_seg, false, dev, &plan_k.use);
    if (st != TA_OK) return st;
  }
  const DeviceWorkList* wk = &plan_k.use.wl;

  const size_t rows = (size_t)B * H * ((size_t)F * T + P);
  const size_t bytes = rows * 2 * sizeof(float) + (size_t)wq->n_slots * part_row +
                       (size_t)wk->n_slots * 2 * part_row;
  void* ws = nullptr;
  st = workspace_for(dev, stream, bytes, &ws);
  if (st != TA_OK) return st;
  float* lse2 = static_cast<float*>(ws);
  float* ndelta = lse2 + rows;
  float* ws_dq = ndelta + rows;
  float* ws_dk = ws_dq + (size_t)wq->n_slots * B * L * d;
  float* ws_dv = ws_dk + (size_t)wk->n_slots * B * L * d;
  const hipStream_t s = static_cast<hipStream_t>(stream);

  ta::PrepArgs pa;
  pa.out = static_cast<const uint16_t*>(out);
  pa.dout = static_cast<const uint16_t*>(dout);
  pa.lse = lse;
  pa.lse2 = lse2;
  pa.ndelta = ndelta;
  pa.rows = (int64_t)rows;
  pa.d = d;
  e = ta::launch_bwd_prep(pa, s);
  if (e != hipSuccess) return fail(TA_ERR_HIP, std::string("prep launch: ") + hipGetErrorString(e));

  ta::BwdArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.dout = static_cast<const uint16_t*>(dout);
  a.dq = static_cast<uint16_t*>(dq);
  a.dk = static_cast<uint16_t*>(dk);
  a.dv = static_cast<uint16_t*>(dv);
  a.B = B;
  a.H = H;
  a.F = F;
  a.T = T;
  a.d = d;
  a.P = P;
  a.lse2 = lse2;
  a.ndelta = ndelta;
  a.items_q = wq->items;
  a.cols_q = wq->cols;
  a.n_items_q = wq->n_items;
  a.ws_dq = ws_dq;
  a.items_k = wk->items;
  a.cols_k = wk->cols;
  a.n_items_k = wk->n_items;
  a.ws_dk = ws_dk;
  a.ws_dv = ws_dv;
  // As in the forward: the logits use |scale| with the sign folded into one
  // operand (q in the dq pass, k in the dk/dv pass); scale 0 zeroes it.
  if (scale == 0.f) {
    a.c = 1.f;
    a.flip = 0u;
    a.keep = 0u;
  } else {
    a.c = std::max(std::fabs(scale) * 1.4426950408889634f, FLT_MIN);
    a.flip = std::signbit(scale) ? 0x80008000u : 0u;
    a.keep = 0xFFFFFFFFu;
  }
  a.scale = scale;
  a.n_wg_q = (uint32_t)((int64_t)B * wq->n_items * nqb);
  a.n_wg_k = (uint32_t)((int64_t)B * wk->n_items * nkb);
  e = ta::launch_bwd_dq(a, s);
  if (e != hipSuccess) return fail(TA_ERR_HIP, std::string("dq launch: ") + hipGetErrorString(e));
  e = ta::launch_bwd_dkdv(a, s);
  if (e != hipSuccess) return fail(TA_ERR_HIP, std::string("dk/dv launch: ") + hipGetErrorString(e));
  auto sum = [&](const DeviceWorkList* wl, const float* part, void* dst, const char* what) -> int {
    if (wl->n_heavy == 0) return TA_OK;
    ta::SumArgs m;
    m.ws = part;
    m.heavy = wl->heavy;
    m.n_heavy = wl->n_heavy;
    m.B = B;
    m.H = H;
    m.F = F;
    m.T = T;
    m.d = d;
    m.P = P;
    m.out = static_cast<uint16_t*>(dst);
    hipError_t err = ta::launch_sum_partials(m, s);
    if (err != hipSuccess)
      return fail(TA_ERR_HIP, std::string(what) + " sum launch: " + hipGetErrorString(err));
    return TA_OK;
  };
  if ((st = sum(wq, ws_dq, dq, "dq")) != TA_OK) return st;
  if ((st = sum(wk, ws_dk, dk, "dk")) != TA_OK) return st;
  if ((st = sum(wk, ws_dv, dv, "dv")) != TA_OK) return st;
  g_last_error.clear();
  return TA_OK;
}

}  // namespace host
}  // namespace ta

using namespace ta::host;

extern "C" {

int tile_attn_make_mask(int F, int k, int form, uint8_t* mask_out) {
  if (!mask_out) return fail(TA_ERR_NULL_PTR, "mask_out must be non-NULL");
  if (F < 1 || F > TA_MAX_FRAMES) return fail(TA_ERR_BAD_SHAPE, "F must be in 1..TA_MAX_FRAMES");
  if (k < 0 || k > F) return fail(TA_ERR_BAD_MASK, "k must be in 0..F");
  if (form != TA_MASK_COL && form != TA_MASK_SYM && form != TA_MASK_DENSE)
    return fail(TA_ERR_BAD_MASK, "unknown mask form");
  std::memset(mask_out, form == TA_MASK_DENSE ? 1 : 0, (size_t)F * F);
  if (form == TA_MASK_DENSE) return TA_OK;
  // Reference frames 0, s, 2s, ... with s = ceil(F / k).
  std::vector<char> is_global(F, 0);
  if (k > 0) {
    const int stride = (F + k - 1) / k;
    for (int j = 0; j < F; j += stride) is_global[j] = 1;
  }
  for (int i = 0; i < F; ++i) {
    uint8_t* row = mask_out + (size_t)i * F;
    const bool full_row = form == TA_MASK_SYM && is_global[i];
    for (int j = 0; j < F; ++j) row[j] = (full_row || i == j || is_global[j]) ? 1 : 0;
  }
  return TA_OK;
}

int tile_attn_compact(const uint8_t* tile_mask, int F, int32_t* row_ptr, uint16_t* cols,
                      uint16_t* order, int* nnz) {
  if (!tile_mask || !row_ptr || !cols || !nnz)
    return fail(TA_ERR_NULL_PTR, "tile_mask, row_ptr, cols and nnz must be non-NULL");
  if (F < 1 || F > TA_MAX_FRAMES) return fail(TA_ERR_BAD_SHAPE, "F must be in 1..TA_MAX_FRAMES");
  compact_host(tile_mask, F, row_ptr, cols, order, nnz);
  return TA_OK;
}

int tile_attn_plan(const uint8_t* tile_mask, int F, int32_t* items, int cap, int* n_items,
                   int* n_slots) {
  if (!tile_mask || !items || !n_items || !n_slots)
    return fail(TA_ERR_NULL_PTR, "tile_mask, items, n_items and n_slots must be non-NULL");
  if (F < 1 || F > TA_MAX_FRAMES) return fail(TA_ERR_BAD_SHAPE, "F must be in 1..TA_MAX_FRAMES");
  const WorkPlan pl = plan_work(tile_mask, F, true);
  *n_items = (int)(pl.items.size() / 4);
  *n_slots = pl.n_slots;
  if (cap < *n_items) return fail(TA_ERR_BAD_SHAPE, "cap is smaller than the number of items");
  std::copy(pl.items.begin(), pl.items.end(), items);
  return TA_OK;
}

int tile_attn_fwd(const void* q, const void* k, const void* v, void* out, int B, int H, int F,
                  int T, int d, const uint8_t* tile_mask, float scale, void* stream) {
  int st = check_args(q, k, v, out, B, H, F, T, d, scale);
  if (st != TA_OK) return st;
  if (!tile_mask) return fail(TA_ERR_NULL_PTR, "tile_mask must be non-NULL");
  return run_fwd(q, k, v, out, B, H, F, T, d, tile_mask, 1, scale, nullptr, stream);
}

int tile_attn_fwd_heads(const void* q, const void* k, const void* v, void* out, int B, int H,
                        int F, int T, int d, const uint8_t* tile_masks, int n_masks, float scale,
                        float* lse, void* stream) {
  int st = check_args(q, k, v, out, B, H, F, T, d, scale);
  if (st != TA_OK) return st;
  if (!tile_masks) return fail(TA_ERR_NULL_PTR, "tile_masks must be non-NULL");
  if (n_masks != 1 && n_masks != H) return fail(TA_ERR_BAD_MASK, "n_masks must be 1 or H");
  if (lse) {
    if (reinterpret_cast<uintptr_t>(lse) % 4) return fail(TA_ERR_ALIGN, "lse must be 4-byte aligned");
    const size_t bytes = (size_t)B * H * F * T * d * 2;
    const size_t lbytes = (size_t)B * H * F * T * sizeof(float);
    for (const void* p : {q, k, v, (const void*)out})
      if (ranges_overlap(lse, lbytes, p, bytes)) return fail(TA_ERR_OVERLAP, "lse overlaps a tensor");
  }
  return run_fwd(q, k, v, out, B, H, F, T, d, tile_masks, n_masks, scale, lse, stream);
}

int tile_attn_fwd_mmdit(const void* q, const void* k, const void* v, void* out, int B, int H,
                        int F, int T, int P, int d, const uint8_t* tile_masks, int n_masks,
                        float scale, float* lse, void* stream) {
  int st = check_args(q, k, v, out, B, H, F, T, d, scale, P);
  if (st != TA_OK) return st;
  if (!tile_masks) return fail(TA_ERR_NULL_PTR, "tile_masks must be non-NULL");
  if (n_masks != 1 && n_masks != H) return fail(TA_ERR_BAD_MASK, "n_masks must be 1 or H");
  if (F + (P > 0) > TA_MAX_FRAMES + 1) return fail(TA_ERR_BAD_SHAPE, "F exceeds TA_MAX_FRAMES");
  if (lse) {
    if (reinterpret_cast<uintptr_t>(lse) % 4) return fail(TA_ERR_ALIGN, "lse must be 4-byte aligned");
    const size_t rows = (size_t)B * H * ((size_t)F * T + P);
    for (const void* p : {q, k, v, (const void*)out})
      if (ranges_overlap(lse, rows * sizeof(float), p, rows * d * 2))
        return fail(TA_ERR_OVERLAP, "lse overlaps a tensor");
  }
  return run_fwd(q, k, v, out, B, H, F, T, d, tile_masks, n_masks, scale, lse, stream, P);
}

int dense_attn_fwd(const void* q, const void* k, const void* v, void* out, int B, int H, int F,
                   int T, int d, float scale, void* stream) {
  int st = check_args(q, k, v, out, B, H, F, T, d, scale);
  if (st != TA_OK) return st;
  std::vector<uint8_t> ones((size_t)F * F, 1);
  return run_fwd(q, k, v, out, B, H, F, T, d, ones.data(), 1, scale, nullptr, stream);
}

}  // extern "C"

namespace {

int check_bwd(const void* q, const void* k, const void* v, const void* out, const void* dout,
              const float* lse, void* dq, void* dk, void* dv, int B, int H, int F, int T, int P,
              int d, const uint8_t* tile_masks, int n_masks, float scale) {
  if (!out || !dout || !lse || !dq || !dk || !dv)
    return fail(TA_ERR_NULL_PTR, "out, dout, lse, dq, dk and dv must be non-NULL");
  int st = check_args(q, k, v, dq, B, H, F, T, d, scale, P);
  if (st != TA_OK) return st;
  if (!tile_masks) return fail(TA_ERR_NULL_PTR, "tile_masks must be non-NULL");
  if (n_masks != 1 && n_masks != H) return fail(TA_ERR_BAD_MASK, "n_masks must be 1 or H");
  for (const void* p : {out, dout, (const void*)dk, (const void*)dv})
    if (reinterpret_cast<uintptr_t>(p) % 16)
      return fail(TA_ERR_ALIGN, "q, k, v, out, dout, dq, dk and dv must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(lse) % 4) return fail(TA_ERR_ALIGN, "lse must be 4-byte aligned");
  const int kpw = ta::bwd_keys_per_workgroup(d), qpw = ta::bwd_queries_per_workgroup(d);
  const int L = std::max(T, P);
  if ((int64_t)B * H * (F + (P > 0)) * ((L + std::min(kpw, qpw) - 1) / std::min(kpw, qpw)) *
          ta::kThreads > (int64_t)UINT32_MAX)
    return fail(TA_ERR_BAD_SHAPE, "the gradient passes would exceed the grid limit");
  const size_t rows = (size_t)B * H * ((size_t)F * T + P);
  const size_t bytes = rows * d * 2;
  const size_t lbytes = rows * sizeof(float);
  const void* outs[3] = {dq, dk, dv};
  for (int i = 0; i < 3; ++i) {
    for (const void* p : {q, k, v, out, dout})
      if (ranges_overlap(outs[i], bytes, p, bytes))
        return fail(TA_ERR_OVERLAP, "dq, dk and dv must not overlap an input");
    if (ranges_overlap(outs[i], bytes, lse, lbytes))
      return fail(TA_ERR_OVERLAP, "dq, dk and dv must not overlap lse");
    for (int j = i + 1; j < 3; ++j)
      if (ranges_overlap(outs[i], bytes, outs[j], bytes))
        return fail(TA_ERR_OVERLAP, "dq, dk and dv must not overlap each other");
  }
  return TA_OK;
}

}  // namespace

extern "C" {

int tile_attn_bwd(const void* q, const void* k, const void* v, const void* out, const void* dout,
                  const float* lse, void* dq, void* dk, void* dv, int B, int H, int F, int T, int d,
                  const uint8_t* tile_masks, int n_masks, float scale, void* stream) {
  const int st = check_bwd(q, k, v, out, dout, lse, dq, dk, dv, B, H, F, T, 0, d, tile_masks,
                           n_masks, scale);
  if (st != TA_OK) return st;
  return run_bwd(q, k, v, out, dout, lse, dq, dk, dv, B, H, F, T, d, tile_masks, n_masks, scale,
                 stream);
}

int tile_attn_bwd_mmdit(const void* q, const void* k, const void* v, const void* out,
                        const void* dout, const float* lse, void* dq, void* dk, void* dv, int B,
                        int H, int F, int T, int P, int d, const uint8_t* tile_masks, int n_masks,
                        float scale, void* stream) {
  const int st = check_bwd(q, k, v, out, dout, lse, dq, dk, dv, B, H, F, T, P, d, tile_masks,
                           n_masks, scale);
  if (st != TA_OK) return st;
  return run_bwd(q, k, v, out, dout, lse, dq, dk, dv, B, H, F, T, d, tile_masks, n_masks, scale,
                 stream, P);
}

const char* tile_attn_status_string(int status) {
  switch (status) {
    case TA_OK: return "ok";
    case TA_ERR_NULL_PTR: return "null pointer";
    case TA_ERR_BAD_SHAPE: return "bad shape";
    case TA_ERR_HEAD_DIM: return "unsupported head dimension";
    case TA_ERR_BAD_MASK: return "bad mask recipe";
    case TA_ERR_ALIGN: return "misaligned pointer";
    case TA_ERR_BAD_SCALE: return "non-finite scale";
    case TA_ERR_OVERLAP: return "output overlaps an input";
    case TA_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

const char* tile_attn_last_error(void) { return g_last_error.c_str(); }

int tile_attn_plan_cache_stats(int* live, int* retired) {
  if (!live || !retired) return fail(TA_ERR_NULL_PTR, "live and retired must be non-NULL");
  std::lock_guard<std::mutex> lock(g_cache_mutex);
  g_cache.collect();
  *live = (int)g_cache.size();
  *retired = (int)g_cache.retired();
  return TA_OK;
}

}  // extern "C"
