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
// Pipeline (one barrier per 64-key tile t)
//   global loads of K(t+2) and V(t+1) are in flight while the wave computes
//   S(t+1) = K(t+1) Q^T on the matrix cores and the softmax of S(t) on the
//   vector ALUs (independent work the two units overlap), then O^T += V(t)^T P(t)^T.
//   K and V each have two LDS buffers; K runs one tile ahead of V.
//
// Online softmax (fp32, base 2): logits are scaled by c = |scale| * log2(e).
// The exponent reference m_ref is only raised when a tile's max exceeds it by
// more than 2^kLazyLog2 in weight; in between, weights may reach 2^kLazyLog2,
// which fp32 and bf16 hold exactly as well as weights <= 1, and the rescale of
// O^T and l is skipped. The result is the same softmax; only the reference of
// the exponentials moves less often. The row sum l is accumulated from the
// bf16-rounded weights that also feed the PV product.
#include <hip/hip_runtime.h>

#include <float.h>
#include <stdint.h>

#include "launch.h"

namespace ta {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWaves = kThreads / 64;
constexpr int kWaveQ = 32;   // query rows per wave: the N side of the 32x32 MFMA
constexpr int kBlockK = 64;  // keys per K/V tile staged in LDS
constexpr float kLazyLog2 = 8.f;
static_assert(kWaves * kWaveQ == kBlockQ, "workgroup rows");

template <int D>
struct Shape {
  static constexpr int kStrideK = D + 8;        // LDS row stride of a K tile (bf16)
  static constexpr int kStrideV = kBlockK + 8;  // LDS row stride of a V^T tile (bf16)
  static constexpr int kChunks = D / 16;        // 16-wide slices of the QK^T contraction
  static constexpr int kDBlocks = D / 32;       // 32-row blocks of O^T
  static constexpr int kKVecs = kBlockK * D / 8;            // 16-byte pieces of a K tile
  static constexpr int kKPerThread = (kKVecs + kThreads - 1) / kThreads;
  static constexpr int kVGroups = (kBlockK / 4) * (D / 8);  // 4-key x 8-d pieces of a V tile
  static_assert(kVGroups <= kThreads, "one V piece per thread");
  static constexpr int kSizeK = kBlockK * kStrideK;
  static constexpr int kSizeV = D * kStrideV;
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

// Position of a group of 4 keys (index kg within the 64-key tile) inside a
// transposed V row. Each 16-key chunk is stored as keys 0-3, 8-11, 4-7, 12-15,
// so the eight keys lane half h contracts over (4h..4h+3 and 8+4h..8+4h+3, the
// C-layout rows it owns) are contiguous.
__device__ __forceinline__ int vt_pos(int kg) {
  return (kg >> 2) * 16 + ((kg & 1) << 3) + ((kg & 2) << 1);
}

// Walks the kept tiles of one query frame in order: tile (e, kt) covers keys
// [64*kt, 64*kt + 64) of kept frame cols[e]. All state is wave-uniform (SGPRs);
// the kept list is read with one scalar load per kept frame.
struct TileCursor {
  const int32_t* cols;  // kept frames of this query frame
  int e = 0, kt = 0, kf = 0;
  int tiles_per_frame, T;
  __device__ __forceinline__ void start(const int32_t* c, int tpf, int t_len, int skip) {
    cols = c;
    tiles_per_frame = tpf;
    T = t_len;
    e = skip / tpf;
    kt = skip % tpf;
    kf = cols[e];
  }
  __device__ __forceinline__ void advance(int n_frames) {
    if (++kt == tiles_per_frame) {
      kt = 0;
      if (++e < n_frames) kf = cols[e];
    }
  }
  __device__ __forceinline__ size_t key0() const { return (size_t)kf * T + kt * kBlockK; }
  __device__ __forceinline__ int nvalid() const { return min(kBlockK, T - kt * kBlockK); }
};

// Buffer resource over the valid rows of one tile: loads past nvalid rows return
// zero (hardware range check), so tiles never read beyond their frame.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const uint16_t* base, int nvalid,
                                                            int d) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(base), (short)0,
                                           nvalid * d * 2, 0x00020000);
}

__device__ __forceinline__ u32x4 buf_load16(__amdgpu_buffer_rsrc_t r, int byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0);
}

// Both halves of the wave see max/sum over lanes l and l^32 (v_permlane32_swap
// hands each lane its partner's value).
__device__ __forceinline__ float pair_max(float x) {
  const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(s[0]), __uint_as_float(s[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}

template <int D>
struct KStage {
  static_assert(Shape<D>::kKVecs % kThreads == 0, "whole K pieces per thread");
  u32x4 r[Shape<D>::kKPerThread];
  __device__ __forceinline__ void load(const uint16_t* Kh, size_t key0, int nvalid, int tid) {
    const __amdgpu_buffer_rsrc_t rs = tile_rsrc(Kh + key0 * D, nvalid, D);
#pragma unroll
    for (int i = 0; i < Shape<D>::kKPerThread; ++i) {
      const int idx = tid + i * kThreads;
      const int row = idx / (D / 8), c8 = idx % (D / 8);
      r[i] = buf_load16(rs, (row * D + 8 * c8) * 2);
    }
  }
  __device__ __forceinline__ void store(uint16_t* sK, int tid) const {
#pragma unroll
    for (int i = 0; i < Shape<D>::kKPerThread; ++i) {
      const int idx = tid + i * kThreads;
      const int row = idx / (D / 8), c8 = idx % (D / 8);
      *reinterpret_cast<u32x4*>(sK + row * Shape<D>::kStrideK + 8 * c8) = r[i];
    }
  }
};

template <int D>
struct VStage {
  u32x4 r[4];  // 4 consecutive keys x 8 consecutive d
  // Threads past kVGroups (whole waves) stage nothing.
  __device__ __forceinline__ void load(const uint16_t* Vh, size_t key0, int nvalid, int tid) {
    if (tid >= Shape<D>::kVGroups) return;
    const int kg = tid % (kBlockK / 4), dg = tid / (kBlockK / 4);
    const __amdgpu_buffer_rsrc_t rs = tile_rsrc(Vh + key0 * D, nvalid, D);
#pragma unroll
    for (int j = 0; j < 4; ++j) r[j] = buf_load16(rs, ((4 * kg + j) * D + 8 * dg) * 2);
  }
  // Transpose 4 keys x 8 d into 8 rows of V^T (4 keys = 8 bytes each).
  __device__ __forceinline__ void store(uint16_t* sV, int tid) const {
    if (tid >= Shape<D>::kVGroups) return;
    const int kg = tid % (kBlockK / 4), dg = tid / (kBlockK / 4);
    const int pos = vt_pos(kg);
#pragma unroll
    for (int mm = 0; mm < 4; ++mm) {
      u32x2 lo, hi;
      lo[0] = __builtin_amdgcn_perm(r[1][mm], r[0][mm], 0x05040100u);
      lo[1] = __builtin_amdgcn_perm(r[3][mm], r[2][mm], 0x05040100u);
      hi[0] = __builtin_amdgcn_perm(r[1][mm], r[0][mm], 0x07060302u);
      hi[1] = __builtin_amdgcn_perm(r[3][mm], r[2][mm], 0x07060302u);
      *reinterpret_cast<u32x2*>(sV + (8 * dg + 2 * mm) * Shape<D>::kStrideV + pos) = lo;
      *reinterpret_cast<u32x2*>(sV + (8 * dg + 2 * mm + 1) * Shape<D>::kStrideV + pos) = hi;
    }
  }
};

// S^T (64 keys x 32 queries) = K_tile * Q^T. In a frame's last tile the keys past
// the frame end start from -inf, so they drop out of the max and get weight 0.
template <int D>
__device__ __forceinline__ void qk_tile(const uint16_t* sK, const bf16x8 (&qf)[D / 16], int n,
                                        int hf, int nvalid, f32x16 (&s)[2]) {
  if (nvalid < kBlockK) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kb * 32 + 8 * (r >> 2) + 4 * hf + (r & 3);
        s[kb][r] = key < nvalid ? 0.f : -INFINITY;
      }
  } else {
    s[0] = f32x16{};
    s[1] = f32x16{};
  }
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
    for (int cc = 0; cc < D / 16; ++cc) {
      const bf16x8 a =
          as_bf16x8(load16(sK + (kb * 32 + n) * Shape<D>::kStrideK + 16 * cc + 8 * hf));
      s[kb] = mfma32(a, qf[cc], s[kb]);
    }
  }
}

// O^T (d x 32 queries) += V_tile^T * P^T.
template <int D>
__device__ __forceinline__ void pv_tile(const uint16_t* sV, const bf16x8 (&pf)[4], int n, int hf,
                                        f32x16 (&o)[D / 32]) {
#pragma unroll
  for (int ch = 0; ch < 4; ++ch)
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb) {
      const bf16x8 a =
          as_bf16x8(load16(sV + (mb * 32 + n) * Shape<D>::kStrideV + 16 * ch + 8 * hf));
      o[mb] = mfma32(a, pf[ch], o[mb]);
    }
}

// Online softmax of one 64-key tile of S^T: updates the running state and
// returns the bf16 weights in B-operand form (chunk ch = accumulator entries
// 8*(ch%2)..+7 of key block ch/2, exactly this lane's 8 keys of that chunk).
// c > 0 always (the host passes a tiny positive c for scale 0), so masked keys
// (-inf) map to exp2(-inf) = 0.
template <int D>
__device__ __forceinline__ void softmax_tile(f32x16 (&s)[2], float c, float lazy_raw,
                                             float& m_ref, float& l_run, f32x16 (&o)[D / 32],
                                             bf16x8 (&pf)[4]) {
  float mx = fmaxf(s[0][0], s[0][1]);
#pragma unroll
  for (int r = 2; r < 16; r += 2) mx = fmaxf(fmaxf(mx, s[0][r]), s[0][r + 1]);
#pragma unroll
  for (int r = 0; r < 16; r += 2) mx = fmaxf(fmaxf(mx, s[1][r]), s[1][r + 1]);
  mx = pair_max(mx);

  // Raise the exponent reference only when some lane's weights would exceed 2^kLazyLog2.
  if (__builtin_amdgcn_ballot_w64(mx - m_ref > lazy_raw) != 0) {
    const float m_new = fmaxf(m_ref, mx);
    const float alpha = fast_exp2((m_ref - m_new) * c);
    l_run *= alpha;
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb) o[mb] *= alpha;
    m_ref = m_new;
  }
  const float mc = m_ref * c;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int r = 0; r < 16; ++r) s[kb][r] = fast_exp2(__builtin_fmaf(s[kb][r], c, -mc));
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  float ls = 0.f;
#pragma unroll
  for (int ch = 0; ch < 4; ++ch) {
    const f32x16& sb = s[ch >> 1];
    const int base = 8 * (ch & 1);
    f32x8 x = {sb[base + 0], sb[base + 1], sb[base + 2], sb[base + 3],
               sb[base + 4], sb[base + 5], sb[base + 6], sb[base + 7]};
    pf[ch] = __builtin_convertvector(x, bf16x8);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bf16x2 pair = {pf[ch][2 * e], pf[ch][2 * e + 1]};
      ls = __builtin_amdgcn_fdot2_f32_bf16(pair, ones, ls, false);
    }
  }
  l_run += pair_sum(ls);
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void tile_attn_fwd_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, uint16_t* __restrict__ O,
    const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ cols,
    const int32_t* __restrict__ order, int F, int T, int nqb, uint32_t n_wg, float c,
    uint32_t qflip, uint32_t qmask) {
  using Sh = Shape<D>;
  __shared__ __attribute__((aligned(16))) uint16_t sK[2][Sh::kSizeK];
  __shared__ __attribute__((aligned(16))) uint16_t sV[2][Sh::kSizeV];

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
  // Waves whose 32 rows all lie past the frame end only help stage tiles.
  const bool wave_active = qb * kBlockQ + wave * kWaveQ < T;
  bf16x8 qf[Sh::kChunks];
  {
    const uint16_t* qp = Qh + ((size_t)frame * T + qrow) * D + 8 * hf;
#pragma unroll
    for (int cc = 0; cc < Sh::kChunks; ++cc) {
      u32x4 x = {0u, 0u, 0u, 0u};
      if (qvalid) x = (load16(qp + 16 * cc) & qmask) ^ qflip;
      qf[cc] = as_bf16x8(x);
    }
  }

  f32x16 o[Sh::kDBlocks];
#pragma unroll
  for (int mb = 0; mb < Sh::kDBlocks; ++mb) o[mb] = f32x16{};
  float m_ref = -FLT_MAX;  // exponent reference (raw logit units) of this lane's query
  float l_run = 0.f;       // running sum of weights
  const float lazy_raw = kLazyLog2 / c;

  const int kbeg = row_ptr[frame];
  const int n_kept = row_ptr[frame + 1] - kbeg;
  const int tpf = (T + kBlockK - 1) / kBlockK;
  const int n_tiles = n_kept * tpf;

  if (n_tiles > 0) {
    KStage<D> kst;
    VStage<D> vst;
    // kc points at tile t + 2 (next K to stage), vc at tile t + 1 (next V to stage).
    TileCursor kc, vc;
    kc.start(cols + kbeg, tpf, T, 0);
    kst.load(Kh, kc.key0(), kc.nvalid(), tid);
    vst.load(Vh, kc.key0(), kc.nvalid(), tid);
    const int nv0 = kc.nvalid();
    kst.store(sK[0], tid);
    vst.store(sV[0], tid);
    vc = kc;
    vc.advance(n_kept);
    if (n_tiles > 1) {
      kc.advance(n_kept);
      kst.load(Kh, kc.key0(), kc.nvalid(), tid);
      kst.store(sK[1], tid);
    }
    kc.advance(n_kept);
    __syncthreads();

    f32x16 sa[2], sb[2];
    if (wave_active) qk_tile<D>(sK[0], qf, n, hf, nv0, sa);

    // One pipeline step: softmax + PV of tile t (scores in s_cur), QK^T of
    // tile t + 1 (into s_nxt), staging of K(t+2) and V(t+1).
    auto step = [&](int t, f32x16(&s_cur)[2], f32x16(&s_nxt)[2]) {
      const bool have_k2 = t + 2 < n_tiles, have_v1 = t + 1 < n_tiles;
      if (have_k2) kst.load(Kh, kc.key0(), kc.nvalid(), tid);
      if (have_v1) vst.load(Vh, vc.key0(), vc.nvalid(), tid);
      if (wave_active) {
        if (have_v1) qk_tile<D>(sK[(t + 1) & 1], qf, n, hf, vc.nvalid(), s_nxt);
        bf16x8 pf[4];
        softmax_tile<D>(s_cur, c, lazy_raw, m_ref, l_run, o, pf);
        pv_tile<D>(sV[t & 1], pf, n, hf, o);
      }
      if (have_k2) kst.store(sK[t & 1], tid);
      if (have_v1) vst.store(sV[(t + 1) & 1], tid);
      kc.advance(n_kept);
      vc.advance(n_kept);
      __syncthreads();
    };

    int t = 0;
    for (; t + 1 < n_tiles; t += 2) {
      step(t, sa, sb);
      step(t + 1, sb, sa);
    }
    if (t < n_tiles) step(t, sa, sb);
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
                     a.v, a.out, a.row_ptr, a.cols, a.order, a.F, a.T, nqb, a.n_wg, a.c, a.qflip,
                     a.qmask);
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
