// Host-side pieces shared by the C-ABI translation units: error reporting, argument
// checks, the work plan in host and device form, and the enqueue of the forward
// kernels for a given plan and partial-result buffer.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

namespace ta {
namespace host {

// Records the detail for tile_attn_last_error() and returns status.
int fail(int status, const std::string& detail);
void clear_error();

// Checks shared by every forward entry point (TA_OK or an error status with its
// detail recorded); nothing touches the GPU.
int check_args(const void* q, const void* k, const void* v, void* out, int B, int H, int F,
               int T, int d, float scale, int P = 0);
bool ranges_overlap(const void* a, size_t na, const void* b, size_t nb);

// The work plans of all heads resident on one device: [items][cols][heavy] in int32
// words, read by the kernels with scalar loads. Items are {head, frame, first kept
// entry, count, slot} with cols and slots offset per head; heavy entries are
// {head, frame, first slot, slots}.
// A forward plan also carries its launch schedule (FwdArgs::sched_*).
struct DeviceWorkList {
  void* buffer = nullptr;
  const int32_t* items = nullptr;
  const int32_t* cols = nullptr;
  const int32_t* heavy = nullptr;
  int n_items = 0, n_heavy = 0, n_slots = 0;
  const int32_t* sched_xcd = nullptr;
  const int32_t* cut_units = nullptr;
  int n_cut_units = 0, n_part_slots = 0, wg_per_xcd = 0;
  bool unit_table = false;  // every position is a table entry (no contiguous whole units)
};

// The same plan as host words, before upload: offsets of the parts in words.
struct HostWorkList {
  std::vector<int32_t> words;
  size_t off_cols = 0, off_heavy = 0;
  int n_items = 0, n_heavy = 0, n_slots = 0;
  size_t off_xcd = 0, off_pieces = 0, off_cut_units = 0;
  int n_cut_units = 0, n_part_slots = 0, wg_per_xcd = 0;
  bool unit_table = false;
};

// Workgroups a forward launch keeps resident per XCD (two per compute unit).
int resident_slots_per_xcd(int dev);

// Appends the forward launch schedule to hw (see FwdArgs::sched): B batch entries, nqb
// query blocks of `rows` rows per segment, head dimension d, T tokens per frame and P
// text tokens.
// With share_tail, each XCD whose run would end in a ragged round of whole units (of
// slots_x resident workgroups) runs that round's units in parts over the kept tiles
// instead, one workgroup per part, merged by log-sum-exp; otherwise every unit is one
// workgroup. With by_length, a plan that splits no frame and whose units with rows are
// not already longest first in every XCD's share runs each share longest first (table
// entries for every unit; query blocks past their segment's end are left out).
void append_fwd_schedule(HostWorkList& hw, int B, int nqb, int rows, int d, int T, int P, int F,
                         int slots_x, bool share_tail, bool by_length = false);

// Plans H heads with n_masks masks (1: shared, H: one per head) of F segments; heavy
// query frames are split into pieces when allow_split.
HostWorkList build_work_list(const uint8_t* masks, int n_masks, int H, int F, bool allow_split);

// The device view of hw's words placed at buf.
DeviceWorkList place_work_list(const HostWorkList& hw, void* buf);

// Enqueues the forward kernel (and the merges of split frames and of parts) on stream
// for a plan already resident on the device; ws holds n_slots * B * max(T, P) * (d + 1)
// floats, then n_part_slots * rows * (d + 4) (unused when the plan has neither). queue:
// null for one workgroup per unit, else 9 int32 on the device, zero, that the kernel's
// persistent work loop (d = 64) uses and leaves zero; launches that may run at the same
// time need different queues. slots_x: resident workgroups per XCD.
int enqueue_fwd(const void* q, const void* k, const void* v, void* out, int B, int H, int F,
                int T, int d, int P, const DeviceWorkList& plan, float* ws, float scale,
                float* lse, void* stream, int* queue, int slots_x);

// The forward queue counters of (dev, stream): allocated and zeroed on first use.
int queue_for(int dev, void* stream, int** out);

}  // namespace host
}  // namespace ta
