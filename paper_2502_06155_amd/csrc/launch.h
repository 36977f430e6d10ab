// Internal interface between the C-ABI host code and the gfx950 kernels.
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace ta {

// Query rows per workgroup; each of the four waves owns 64 query rows.
constexpr int kBlockQ = 256;
constexpr int kThreads = 256;

struct FwdArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* out;
  int B, H, F, T, d;
  // Work items, 5 int32 each, in dispatch order: {head, query frame, first kept
  // entry in cols, number of kept entries, partial slot or -1}. Every batch entry
  // runs every item. A query frame with many kept frames is split into several
  // items (slots >= 0) whose partial results the merge kernel combines; every
  // other frame is one item (slot -1) that writes out directly.
  const int32_t* items;
  const int32_t* cols;  // kept key frames, row after row, head after head
  int n_items;          // items over all heads
  float* ws_o;          // partial O/l, fp32 [n_slots][B][T][d] (null if no slots)
  float* ws_lse;        // partial base-2 log-sum-exp, fp32 [n_slots][B][T]
  float* lse;           // natural-log log-sum-exp out, fp32 [B][H][F*T], or null
  float c;              // > 0: |scale| * log2(e), logits in base-2 units
  uint32_t qflip;       // 0x80008000 flips the sign of q (negative scale), else 0
  uint32_t qmask;       // 0 zeroes q (scale 0: exactly uniform weights), else ~0
  uint32_t n_wg;        // B * n_items * ceil(T / kBlockQ)
};

// Combines the partial results of split query frames: heavy holds 4 int32 per split
// frame {head, query frame, first slot, number of slots}.
struct MergeArgs {
  const float* ws_o;
  const float* ws_lse;
  const int32_t* heavy;
  int n_heavy;
  int B, H, F, T, d;
  uint16_t* out;
  float* lse;  // natural-log log-sum-exp out or null
};

hipError_t launch_tile_attn_fwd(const FwdArgs& a, hipStream_t stream);
hipError_t launch_merge_partials(const MergeArgs& a, hipStream_t stream);

}  // namespace ta
