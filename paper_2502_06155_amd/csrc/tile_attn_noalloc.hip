// tile_attn_fwd_heads_noalloc: the forward of tile_attn_fwd_heads for callers that
// cannot allocate device memory (code being captured into a graph, tight serving
// loops, harnesses that forbid allocation). The work plan and the partial results of
// split query frames live in one static device array per GPU instead of the cached
// plan buffers and per-stream workspaces of the other entry points; the plan words
// travel to it by value, in the arguments of small store kernels, so a call enqueues
// only kernel launches and never reads host memory after it returns.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <map>
#include <mutex>
#include <string>

#include "../../include/tile_attn.h"
#include "host_internal.h"
#include "launch.h"

namespace {

constexpr size_t kPlanWords = TA_NOALLOC_PLAN_WORDS;
constexpr size_t kPartialFloats = TA_NOALLOC_PARTIAL_BYTES / sizeof(float);
static_assert(kPlanWords % 64 == 0, "the partial results start 256-byte aligned");

// [plan words][partial O/l and log-sum-exp of split frames]. Each GPU holds its own
// copy from the moment the library's code is loaded on it until the process ends.
static __device__ __align__(256) int32_t scratch[kPlanWords + kPartialFloats];

// Plan words carried by one store launch, by value in its kernel arguments (kept
// under the 4 KiB kernel-argument limit).
constexpr int kWordsPerStore = 960;
struct StoreArgs {
  int32_t* dst;
  int n;
  int32_t w[kWordsPerStore];
};

__global__ __launch_bounds__(256) void store_words_kernel(StoreArgs a) {
  for (int i = threadIdx.x; i < a.n; i += 256) a.dst[i] = a.w[i];
}

// Device address of `scratch` per device, looked up once per device with that device
// current (each device has its own copy of the array at its own address). Host code
// uses only these addresses: the array's name in host code is not a device address.
std::mutex g_scratch_mutex;
std::map<int, int32_t*> g_scratch;

int scratch_on(int dev, int32_t** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  auto it = g_scratch.find(dev);
  if (it == g_scratch.end()) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return ta::host::fail(TA_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") +
                                            hipGetErrorString(e));
    it = g_scratch.emplace(dev, static_cast<int32_t*>(p)).first;
  }
  *out = it->second;
  return TA_OK;
}

}  // namespace

extern "C" int tile_attn_fwd_heads_noalloc(const void* q, const void* k, const void* v, void* out,
                                           int B, int H, int F, int T, int d,
                                           const uint8_t* tile_masks, int n_masks, float scale,
                                           float* lse, void* stream) {
  using namespace ta::host;
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
  // The plan: heavy frames split as in tile_attn_fwd_heads when their partial results
  // fit the scratch array, otherwise every frame in one piece (no partials).
  const int64_t nqb = (T + ta::fwd_rows_per_workgroup(d) - 1) / ta::fwd_rows_per_workgroup(d);
  const int64_t max_wg = (int64_t)UINT32_MAX / ta::kThreads;
  // Every unit runs whole (no shared-out tail): the partials stay those of split frames.
  const int rows = ta::fwd_rows_per_workgroup(d);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  const int slots_x = e == hipSuccess ? resident_slots_per_xcd(dev) : 64;
  HostWorkList hw = build_work_list(tile_masks, n_masks, H, F, true);
  if ((size_t)hw.n_slots * B * T * (d + 1) > kPartialFloats || (int64_t)B * hw.n_items * nqb > max_wg)
    hw = build_work_list(tile_masks, n_masks, H, F, false);
  append_fwd_schedule(hw, B, (int)nqb, rows, d, T, 0, F, slots_x, false);
  if (hw.words.size() > kPlanWords)
    return fail(TA_ERR_BAD_SHAPE, "the work plan needs " + std::to_string(hw.words.size()) +
                                      " words, more than the " + std::to_string(kPlanWords) +
                                      " of tile_attn_fwd_heads_noalloc's static scratch");
  if (e != hipSuccess) return fail(TA_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  int32_t* base = nullptr;
  if ((st = scratch_on(dev, &base)) != TA_OK) return st;

  const hipStream_t s = static_cast<hipStream_t>(stream);
  for (size_t off = 0; off < hw.words.size(); off += kWordsPerStore) {
    StoreArgs a;
    a.dst = base + off;
    a.n = (int)std::min<size_t>(kWordsPerStore, hw.words.size() - off);
    std::copy(hw.words.begin() + off, hw.words.begin() + off + a.n, a.w);
    hipLaunchKernelGGL(store_words_kernel, dim3(1), dim3(256), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess)
      return fail(TA_ERR_HIP, std::string("plan store launch: ") + hipGetErrorString(e));
  }
  const DeviceWorkList wl = place_work_list(hw, base);
  float* partials = reinterpret_cast<float*>(base + kPlanWords);
  // No text prefix here, so one workgroup per unit (no work-queue counters).
  st = enqueue_fwd(q, k, v, out, B, H, F, T, d, 0, wl, partials, scale, lse, stream, nullptr, slots_x);
  if (st != TA_OK) return st;
  clear_error();
  return TA_OK;
}
