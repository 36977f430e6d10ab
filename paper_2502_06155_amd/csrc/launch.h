// Internal interface between the C-ABI host code and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace ta {

constexpr int kThreads = 256;

// Query rows per forward workgroup for head dimension d (4 waves of 64 rows, or of 32
// rows at d = 128).
int fwd_rows_per_workgroup(int d);

struct FwdArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* out;
  int B, H, F, T, d;
  // Text tokens before the F*T video tokens (MM-DiT form), or 0. With P > 0 the
  // work items address F + 1 segments: frames 0..F-1 at P + j*T, the text as F.
  int P;
  // Work items, 5 int32 each, in dispatch order: {head, query frame, first kept
  // entry in cols, number of kept entries, partial slot or -1}. Every batch entry
  // runs every item. A query frame with many kept frames is split into several
  // items (slots >= 0) whose partial results the merge kernel combines; every
  // other frame is one item (slot -1) that writes out directly.
  const int32_t* items;
  const int32_t* cols;  // kept key frames, row after row, head after head
  int n_items;          // items over all heads
  float* ws_o;          // partial O/l, fp32 [n_slots][B][max(T,P)][d] (null if no slots)
  float* ws_lse;        // partial base-2 log-sum-exp, fp32 [n_slots][B][max(T,P)]
  float* lse;           // natural-log log-sum-exp out, fp32 [B][H][P+F*T], or null
  float c;              // > 0: |scale| * log2(e), logits in base-2 units
  uint32_t qflip;       // 0x80008000 flips the sign of q (negative scale), else 0
  uint32_t qmask;       // 0 zeroes q (scale 0: exactly uniform weights), else ~0
  // The launch schedule (on the device): per XCD (8 of them) {first unit, contiguous
  // whole units, table entries, first entry}, then the table entries {unit, first
  // tile, tiles, partial slot (-1: a whole unit)}; and per unit run in parts {unit,
  // first partial slot, parts}. Units are (b, item, query block), query block fastest.
  const int32_t* sched;
  const int32_t* cut_units;
  int n_cut_units;
  int wg_per_xcd;       // queue positions of the busiest XCD
  bool unit_table;      // every position is a piece of the table (none contiguous)
  int slots_per_xcd;    // resident workgroups per XCD: the grid is 8 * min(that, wg_per_xcd)
  // Work-queue counters for the persistent form of the kernel (9 int32 on the device,
  // zero between launches: the kernel resets them), or null for one workgroup per unit.
  // Used at d = 64 only.
  int* queue;
  float* ws_parts;         // parts, fp32 [slot][fwd_rows_per_workgroup(d)][d + 4]: O/l, log-sum-exp
};

// Combines the partial results of split query frames: heavy holds 4 int32 per split
// frame {head, query frame, first slot, number of slots}.
struct MergeArgs {
  const float* ws_o;
  const float* ws_lse;
  const int32_t* heavy;
  int n_heavy;
  int B, H, F, T, d;
  int P;       // text tokens before the video (0: none)
  uint16_t* out;
  float* lse;  // natural-log log-sum-exp out or null
};

hipError_t launch_tile_attn_fwd(const FwdArgs& a, hipStream_t stream);
hipError_t launch_merge_partials(const MergeArgs& a, hipStream_t stream);

// Gradients. The prep pass turns the forward's natural-log log-sum-exp into base 2
// and forms ndelta = -<dO, out> per query row (negated: both gradient kernels start
// their dP accumulations at it, so dP - delta comes out of the matrix cores).
struct PrepArgs {
  const uint16_t* out;
  const uint16_t* dout;
  const float* lse;  // natural log, [rows]
  float* lse2;       // base 2, [rows]
  float* ndelta;     // [rows]
  int64_t rows;      // B * H * F * T
  int d;
};

// The two gradient kernels. The query-side pass (dq) walks each query frame's kept
// key frames with the forward's work list; the key-side pass (dk, dv) walks each
// key frame's keeping query frames with the work list of the transposed mask.
// Items are 5 int32 as in FwdArgs; split frames write fp32 partials [n_slots][B][T][d]
// that sum_partials adds up.
struct BwdArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* dout;
  uint16_t* dq;
  uint16_t* dk;
  uint16_t* dv;
  int B, H, F, T, d;
  int P;  // text tokens before the video (0: none); segments as in FwdArgs
  const float* lse2;
  const float* ndelta;
  const int32_t* items_q;
  const int32_t* cols_q;
  int n_items_q;
  float* ws_dq;
  const int32_t* items_k;
  const int32_t* cols_k;
  int n_items_k;
  float* ws_dk;
  float* ws_dv;
  float c;           // > 0: |scale| * log2(e)
  float scale;       // multiplies dq and dk
  uint32_t flip;     // 0x80008000 flips the sign of the logits' q (dq pass) or k (dk/dv pass)
  uint32_t keep;     // 0 zeroes that operand (scale 0), else ~0
  uint32_t n_wg_q;   // B * n_items_q * ceil(max(T, P) / bwd_queries_per_workgroup(d))
  uint32_t n_wg_k;   // B * n_items_k * ceil(max(T, P) / bwd_keys_per_workgroup(d))
};

// Adds the partials of split segments: heavy holds {head, segment, first slot, slots}.
struct SumArgs {
  const float* ws;
  const int32_t* heavy;
  int n_heavy;
  int B, H, F, T, d;
  int P;
  uint16_t* out;
};

int bwd_queries_per_workgroup(int d);
int bwd_keys_per_workgroup(int d);
hipError_t launch_bwd_prep(const PrepArgs& a, hipStream_t stream);
hipError_t launch_bwd_dq(const BwdArgs& a, hipStream_t stream);
hipError_t launch_bwd_dkdv(const BwdArgs& a, hipStream_t stream);
hipError_t launch_sum_partials(const SumArgs& a, hipStream_t stream);

}  // namespace ta
