// gfx950 (MI355X, CDNA4) kernels for the tile-sparse 3D attention forward pass.
//
// What is computed (Sec. 3.3 of Efficient-vDiT): for every query token of latent
// frame i, softmax attention over the key tokens of the frames j that the
// frame mask keeps. Frames the mask drops are never read (App. B: empty blocks
// are skipped); the kernel walks a compact kept-frame list per query frame.
//
// Work decomposition
//   One workgroup = 4 waves = 128 query rows of one (batch, head, query frame).
//   Query blocks are frame aligned, so every row of a workgroup shares one kept
//   list. Workgroup ids are remapped so that each XCD (8 per MI355X, each with
//   its own L2) receives a contiguous run of (batch, head) problems, which keeps
//   the K/V of the shared global frames resident in that XCD's L2.
//
// Matrix-core layout (v_mfma_f32_32x32x16_bf16, wave64)
//   A (32 x 16): lane l holds row l%32, k = 8*(l/32) .. +7
//   B (16 x 32): lane l holds col l%32, k = 8*(l/32) .. +7
//   C (32 x 32): lane l holds col l%32, rows 8*i + 4*(l/32) + j at index 4*i + j
//   The kernel computes S^T = K * Q^T (A = K rows from LDS, B = this wave's 32
//   queries held in registers), so each lane owns ONE query and 16 of every 32
//   keys: the softmax row max and row sum are in-lane reductions plus a single
//   exchange with lane l^32. The probabilities P^T then sit exactly where the
//   B operand of O^T += V^T * P^T expects them (contraction over keys), and only
//   V needs a transpose, done once per tile while staging it in LDS.
//
// Online softmax (fp32, base 2): logits are scaled by c = |scale| * log2(e);
// m is the running max of the raw logits, l the running sum of exp2 weights,
// and O^T is rescaled by exp2(c * (m_old - m_new)) whenever m grows.
#include <hip/hip_runtime.h>

#include <float.h>
#include <stdint.h>

#include "launch.h"

namespace ta {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = kThreads / 64;
constexpr int kWaveQ = 32;   // query rows per wave: the N side of the 32x32 MFMA
constexpr int kBlockK = 64;  // keys per K/V tile staged in LDS
static_assert(kWaves * kWaveQ == kBlockQ, "workgroup rows");

template <int D>
struct Shape {
  static constexpr int kStrideK = D + 8;        // LDS row stride of the K tile (bf16)
  static constexpr int kStrideV = kBlockK + 8;  // LDS row stride of the V^T tile (bf16)
  static constexpr int kChunks = D / 16;        // 16-wide slices of the QK^T contraction
  static constexpr int kDBlocks = D / 32;       // 32-row blocks of O^T
  static constexpr int kKVecs = kBlockK * D / 8;            // 16-byte pieces of a K tile
  static constexpr int kVGroups = (kBlockK / 4) * (D / 8);  // 4-key x 8-d pieces of a V tile
};

// Workgroup id -> logical work index such that the ids the hardware sends to
// XCD x (those with id % 8 == x) cover one contiguous logical range.
__device__ __forceinline__ uint32_t xcd_remap(uint32_t id, uint32_t n) {
  const uint32_t q = n / 8, r = n % 8, x = id % 8, pos = id / 8;
  return x * q + (x < r ? x : r) + pos;
}

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 x) { return __builtin_bit_cast(bf16x8, x); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Position of key u (0..15) of a 16-key chunk inside a transposed V row: the
// chunk is stored as keys 0-3, 8-11, 4-7, 12-15, so that the eight keys lane
// half h contracts over (4h..4h+3 and 8+4h..8+4h+3, the C-layout rows it owns)
// are contiguous. Only whole groups of 4 keys are placed, so u % 4 == 0.
__device__ __forceinline__ int vt_pos(int kg) {
  return (kg >> 2) * 16 + ((kg & 1) << 3) + ((kg & 2) << 1);
}

template <int D>
__global__ __launch_bounds__(kThreads) void tile_attn_fwd_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, uint16_t* __restrict__ O,
    const int32_t* __restrict__ row_ptr, const uint16_t* __restrict__ cols,
    const uint16_t* __restrict__ order, int F, int T, int nqb, uint32_t n_wg, float c,
    uint32_t qflip) {
  using Sh = Shape<D>;
  __shared__ __attribute__((aligned(16))) uint16_t sK[kBlockK * Sh::kStrideK];
  __shared__ __attribute__((aligned(16))) uint16_t sV[D * Sh::kStrideV];

  const uint32_t work = xcd_remap(blockIdx.x, n_wg);
  const uint32_t per_bh = (uint32_t)F * (uint32_t)nqb;
  const uint32_t bh = work / per_bh;
  const uint32_t rem = work - bh * per_bh;
  const int frame = order[rem / nqb];
  const int qb = (int)(rem % nqb);

  const size_t head_elems = (size_t)F * T * D;
  const uint16_t* Qh = Q + bh * head_elems;
  const uint16_t* Kh = K + bh * head_elems;
  const uint16_t* Vh = V + bh * head_elems;
  uint16_t* Oh = O + bh * head_elems;

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int n = lane & 31, hf = lane >> 5;

  // This lane's query row (within its frame) and its Q^T B-operand slices.
  const int qrow = qb * kBlockQ + wave * kWaveQ + n;
  const bool qvalid = qrow < T;
  bf16x8 qf[Sh::kChunks];
  {
    const uint16_t* qp = Qh + ((size_t)frame * T + qrow) * D + 8 * hf;
#pragma unroll
    for (int cc = 0; cc < Sh::kChunks; ++cc) {
      u32x4 x = {0u, 0u, 0u, 0u};
      if (qvalid) x = load16(qp + 16 * cc) ^ qflip;
      qf[cc] = as_bf16x8(x);
    }
  }

  f32x16 o[Sh::kDBlocks];
#pragma unroll
  for (int mb = 0; mb < Sh::kDBlocks; ++mb) o[mb] = f32x16{};
  float m_run = -FLT_MAX;  // running max of raw logits for this lane's query
  float l_run = 0.f;       // running sum of exp2 weights

  const int kbeg = row_ptr[frame];
  const int kend = row_ptr[frame + 1];
  const int tiles_per_frame = (T + kBlockK - 1) / kBlockK;
  const int n_tiles = (kend - kbeg) * tiles_per_frame;

  for (int t = 0; t < n_tiles; ++t) {
    const int kf = cols[kbeg + t / tiles_per_frame];
    const int k0 = (t % tiles_per_frame) * kBlockK;
    const int nvalid = min(kBlockK, T - k0);
    const size_t key0 = (size_t)kf * T + k0;

    __syncthreads();  // every wave is done reading the previous tile
    // K tile -> LDS, row-major [key][d]; keys past the frame end read as zero.
    for (int i = tid; i < Sh::kKVecs; i += kThreads) {
      const int r = i / (D / 8), c8 = i % (D / 8);
      u32x4 x = {0u, 0u, 0u, 0u};
      if (r < nvalid) x = load16(Kh + (key0 + r) * D + 8 * c8);
      *reinterpret_cast<u32x4*>(sK + r * Sh::kStrideK + 8 * c8) = x;
    }
    // V tile -> LDS transposed [d][key], 4 keys x 8 d per thread per step.
    for (int g = tid; g < Sh::kVGroups; g += kThreads) {
      const int kg = g % (kBlockK / 4), dg = g / (kBlockK / 4);
      u32x4 rv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = 4 * kg + r;
        rv[r] = u32x4{0u, 0u, 0u, 0u};
        if (key < nvalid) rv[r] = load16(Vh + (key0 + key) * D + 8 * dg);
      }
      const int pos = vt_pos(kg);
#pragma unroll
      for (int mm = 0; mm < 4; ++mm) {
        u32x2 lo, hi;
        lo[0] = __builtin_amdgcn_perm(rv[1][mm], rv[0][mm], 0x05040100u);
        lo[1] = __builtin_amdgcn_perm(rv[3][mm], rv[2][mm], 0x05040100u);
        hi[0] = __builtin_amdgcn_perm(rv[1][mm], rv[0][mm], 0x07060302u);
        hi[1] = __builtin_amdgcn_perm(rv[3][mm], rv[2][mm], 0x07060302u);
        *reinterpret_cast<u32x2*>(sV + (8 * dg + 2 * mm) * Sh::kStrideV + pos) = lo;
        *reinterpret_cast<u32x2*>(sV + (8 * dg + 2 * mm + 1) * Sh::kStrideV + pos) = hi;
      }
    }
    __syncthreads();

    // S^T = K * Q^T for two blocks of 32 keys.
    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      s[kb] = f32x16{};
#pragma unroll
      for (int cc = 0; cc < Sh::kChunks; ++cc) {
        const bf16x8 a =
            as_bf16x8(load16(sK + (kb * 32 + n) * Sh::kStrideK + 16 * cc + 8 * hf));
        s[kb] = mfma32(a, qf[cc], s[kb]);
      }
    }

    // Keys past the frame end take no part in the max (their weights are zeroed below).
    const bool tail = nvalid < kBlockK;
    if (tail) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kb * 32 + 8 * (r >> 2) + 4 * hf + (r & 3);
          if (key >= nvalid) s[kb][r] = -INFINITY;
        }
    }

    float mx = s[0][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = fast_exp2((m_run - m_new) * c);
    const float mc = m_new * c;

    float ls = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = fast_exp2(__builtin_fmaf(s[kb][r], c, -mc));
        s[kb][r] = p;
      }
    if (tail) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = kb * 32 + 8 * (r >> 2) + 4 * hf + (r & 3);
          if (key >= nvalid) s[kb][r] = 0.f;
        }
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) ls += s[kb][r];
    ls += __shfl_xor(ls, 32);
    l_run = l_run * alpha + ls;
    m_run = m_new;
#pragma unroll
    for (int mb = 0; mb < Sh::kDBlocks; ++mb) o[mb] *= alpha;

    // P^T in B-operand form: 16-key chunk ch uses accumulator entries 8*(ch%2)..+7
    // of key block ch/2, which are exactly this lane's 8 keys of that chunk.
    bf16x8 pf[4];
#pragma unroll
    for (int ch = 0; ch < 4; ++ch) {
      const f32x16& sb = s[ch >> 1];
      const int base = 8 * (ch & 1);
      f32x8 x = {sb[base + 0], sb[base + 1], sb[base + 2], sb[base + 3],
                 sb[base + 4], sb[base + 5], sb[base + 6], sb[base + 7]};
      pf[ch] = __builtin_convertvector(x, bf16x8);
    }

    // O^T += V^T * P^T.
#pragma unroll
    for (int ch = 0; ch < 4; ++ch)
#pragma unroll
      for (int mb = 0; mb < Sh::kDBlocks; ++mb) {
        const bf16x8 a =
            as_bf16x8(load16(sV + (mb * 32 + n) * Sh::kStrideV + 16 * ch + 8 * hf));
        o[mb] = mfma32(a, pf[ch], o[mb]);
      }
  }

  // Epilogue: normalise, round to bf16 (RNE), store 4 consecutive d per access.
  if (qvalid) {
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
    uint16_t* op = Oh + ((size_t)frame * T + qrow) * D;
#pragma unroll
    for (int mb = 0; mb < Sh::kDBlocks; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f32x4 x = {o[mb][4 * i + 0] * inv, o[mb][4 * i + 1] * inv, o[mb][4 * i + 2] * inv,
                   o[mb][4 * i + 3] * inv};
        const bf16x4 y = __builtin_convertvector(x, bf16x4);
        *reinterpret_cast<u32x2*>(op + 32 * mb + 8 * i + 4 * hf) = __builtin_bit_cast(u32x2, y);
      }
  }
}

template <int D>
hipError_t launch_d(const FwdArgs& a, hipStream_t stream) {
  const int nqb = (a.T + kBlockQ - 1) / kBlockQ;
  hipLaunchKernelGGL(tile_attn_fwd_kernel<D>, dim3(a.n_wg), dim3(kThreads), 0, stream, a.q, a.k,
                     a.v, a.out, a.row_ptr, a.cols, a.order, a.F, a.T, nqb, a.n_wg, a.c, a.qflip);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_tile_attn_fwd(const FwdArgs& a, hipStream_t stream) {
  switch (a.d) {
    case 64: return launch_d<64>(a, stream);
    case 96: return launch_d<96>(a, stream);
    case 128: return launch_d<128>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ta
