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
  const int32_t* row_ptr;  // device, F + 1
  const int32_t* cols;     // device, nnz: kept key frames, row after row
  const int32_t* order;    // device, F: dispatch order of query frames
  float c;                 // > 0: |scale| * log2(e), logits in base-2 units
  uint32_t qflip;          // 0x80008000 flips the sign of q (negative scale), else 0
  uint32_t qmask;          // 0 zeroes q (scale 0: exactly uniform weights), else ~0
  uint32_t n_wg;           // B * H * F * ceil(T / kBlockQ)
};

hipError_t launch_tile_attn_fwd(const FwdArgs& a, hipStream_t stream);

}  // namespace ta
