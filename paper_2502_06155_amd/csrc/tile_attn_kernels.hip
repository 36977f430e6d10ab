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
//   keys. The probabilities P^T then sit exactly where the B operand of
//   O^T += V^T * P^T expects them, with the contraction index k of chunk ch
//   mapped to keys 16ch + 4h + (0..3) and 16ch + 8 + 4h + (0..3) for lane half h.
//   The V^T operand is read from the untransposed V tile with the LDS transpose
//   load ds_read_b64_tr_b16: inside each 16-lane group, lane i receives element
//   i%4 of the 8-byte rows read by lanes 4k + i/4 (k = 0..3), so when lane j reads
//   V[key0 + j/4][d0 + 4(j%4) .. +3], lane i gets V[key0 .. key0+3][d0 + i].
//
// Pipeline (one barrier per 64-key tile t)
//   Step t stores K(t+2) and V(t+1), loaded into registers during step t-1, into
//   the LDS buffers that tiles t and t-1 freed, and starts the global loads of
//   K(t+3) and V(t+2), which have a whole step to arrive. It then runs in two
//   halves over 32-key blocks: QK^T of a block of tile t+1, the weights of the
//   previous block and PV of the one before, three independent pieces whose
//   MFMAs and VALU work interleave. K and V each have two LDS buffers; K runs one
//   tile ahead of V.
//
// Online softmax (fp32, base 2): weights are exp2(c * (s - m_ref)) with
// c = |scale| * log2(e) and m_ref an exponent reference per query that only
// moves when needed. The first tile sets m_ref to its row max. After that the
// weights are formed directly; if any lane's sum of weights in a tile exceeds
// 2^kLazyLog2 (so some weight may have grown past it), that tile is redone with
// m_ref raised to the running max and O^T and l rescaled. Weights up to
// 2^kLazyLog2 are as exact in fp32 and bf16 as weights up to 1, so the result is
// the same softmax; only the reference of the exponentials moves less often. The
// row sum l is accumulated from the bf16-rounded weights that also feed the PV
// product, per lane (its 16 of every 32 keys) and summed over the two lane
// halves once, in the epilogue.
#include <hip/hip_runtime.h>

#include <float.h>
#include <stdint.h>

#include "launch.h"

namespace ta {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kWaves = kThreads / 64;
constexpr int kWaveQ = 32;   // query rows per wave: the N side of the 32x32 MFMA
constexpr int kBlockK = 64;  // keys per K/V tile staged in LDS
constexpr float kLazyLog2 = 10.f;
static_assert(kWaves * kWaveQ == kBlockQ, "workgroup rows");

template <int D>
struct Shape {
  // LDS row strides (bf16). K rows are read 16 bytes per lane, 16 rows at a time:
  // D + 8 spreads those rows over all 64 banks. V rows are read 8 bytes per lane by
  // the transpose load, 4 rows x 64 bytes at a time: a stride of 48 or 16 banks
  // (mod 64) keeps those four rows apart.
  static constexpr int kStrideK = D + 8;
  static constexpr int kStrideV = (D % 64 == 32) ? D : D + 32;
  static constexpr int kChunks = D / 16;   // 16-wide slices of the QK^T contraction
  static constexpr int kDBlocks = D / 32;  // 32-row blocks of O^T
  static constexpr int kPieces = D / 8;    // 16-byte pieces per K/V row
  static constexpr int kPiecesPerThread = kBlockK * kPieces / kThreads;
  static_assert(kBlockK * kPieces % kThreads == 0, "whole pieces per thread");
  static constexpr int kSizeK = kBlockK * kStrideK;
  static constexpr int kSizeV = kBlockK * kStrideV;
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

// Walks the kept tiles of one query frame in order: tile (e, kt) covers keys
// [64*kt, 64*kt + 64) of kept frame cols[e]. All state is wave-uniform (SGPRs);
// the kept list is read with one scalar load per kept frame.
struct TileCursor {
  const int32_t* cols;  // kept frames of this query frame
  int e = 0, kt = 0, kf = 0;
  int tiles_per_frame, T;
  __device__ __forceinline__ void start(const int32_t* c, int tpf, int t_len) {
    cols = c;
    tiles_per_frame = tpf;
    T = t_len;
    e = 0;
    kt = 0;
    kf = cols[0];
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

// Register staging of one 64-key K or V tile: the tile is kBlockK * D contiguous
// bf16 in global memory, cut into 16-byte pieces; thread tid moves pieces
// tid, tid + 256, ... into LDS rows of the given stride.
template <int D>
struct Stage {
  u32x4 r[Shape<D>::kPiecesPerThread];
  __device__ __forceinline__ void load(const uint16_t* Xh, size_t key0, int nvalid, int tid) {
    const __amdgpu_buffer_rsrc_t rs = tile_rsrc(Xh + key0 * D, nvalid, D);
#pragma unroll
    for (int i = 0; i < Shape<D>::kPiecesPerThread; ++i)
      r[i] = buf_load16(rs, (tid + i * kThreads) * 16);
  }
  template <int STRIDE>
  __device__ __forceinline__ void store(uint16_t* s, int tid) const {
#pragma unroll
    for (int i = 0; i < Shape<D>::kPiecesPerThread; ++i) {
      const int idx = tid + i * kThreads;
      const int row = idx / Shape<D>::kPieces, c8 = idx % Shape<D>::kPieces;
      *reinterpret_cast<u32x4*>(s + row * STRIDE + 8 * c8) = r[i];
    }
  }
};

// S^T of 32-key block kb of a K tile (32 keys x 32 queries), raw logits.
template <int D>
__device__ __forceinline__ f32x16 qk_block(const uint16_t* sK, const bf16x8 (&qf)[D / 16], int n,
                                           int hf, int kb) {
  const uint16_t* row = sK + (kb * 32 + n) * Shape<D>::kStrideK + 8 * hf;
  f32x16 s = mfma32(as_bf16x8(load16(row)), qf[0], f32x16{});
#pragma unroll
  for (int cc = 1; cc < D / 16; ++cc) s = mfma32(as_bf16x8(load16(row + 16 * cc)), qf[cc], s);
  return s;
}

// Keys of block kb past the frame end get -inf: no part in the max, weight 0.
__device__ __forceinline__ void mask_tail(f32x16& s, int kb, int hf, int nvalid) {
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int key = kb * 32 + 8 * (r >> 2) + 4 * hf + (r & 3);
    if (key >= nvalid) s[r] = -INFINITY;
  }
}

// V^T fragment (32 d-rows x 16 keys, A-operand layout) for d-block mb and key
// chunk ch, from a V tile stored row-major (key, d) in LDS. Lane l: group
// g = l/16, j = l%16 reads V[16ch + 4(g/2) + j/4 (+8)][32mb + 16(g%2) + 4(j%4) ..].
template <int D>
__device__ __forceinline__ bf16x8 vt_frag(const uint16_t* sV, int lane, int mb, int ch) {
  const int g = lane >> 4, j = lane & 15;
  const uint16_t* p =
      sV + (16 * ch + 4 * (g >> 1) + (j >> 2)) * Shape<D>::kStrideV + 32 * mb + 16 * (g & 1) + 4 * (j & 3);
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 8 * Shape<D>::kStrideV));
  const u32x2 a = __builtin_bit_cast(u32x2, lo), b = __builtin_bit_cast(u32x2, hi);
  return as_bf16x8(u32x4{a[0], a[1], b[0], b[1]});
}

// O^T (d x 32 queries) += V^T * P^T over 32-key block kb (key chunks 2kb, 2kb+1).
template <int D>
__device__ __forceinline__ void pv_block(const uint16_t* sV, const bf16x8 (&p)[2], int lane, int kb,
                                         f32x16 (&o)[D / 32]) {
#pragma unroll
  for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb)
      o[mb] = mfma32(vt_frag<D>(sV, lane, mb, 2 * kb + c2), p[c2], o[mb]);
}

// This lane's max over its 16 scores of a block (-inf keys included).
__device__ __forceinline__ float block_max(const f32x16& s) {
  float mx = fmaxf(s[0], s[1]);
#pragma unroll
  for (int r = 2; r < 16; r += 2) mx = fmaxf(fmaxf(mx, s[r]), s[r + 1]);
  return mx;
}

// Weights exp2(c*s - mc) of one 32-key block in B-operand form (chunk c2 =
// accumulator entries 8*c2 .. 8*c2+7, exactly this lane's 8 keys of that 16-key
// chunk); returns this lane's sum of the bf16-rounded weights.
__device__ __forceinline__ float block_weights(const f32x16& s, float c, float mc, bf16x8 (&p)[2]) {
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  float ls = 0.f;
#pragma unroll
  for (int c2 = 0; c2 < 2; ++c2) {
    f32x8 x;
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = fast_exp2(__builtin_fmaf(s[8 * c2 + e], c, -mc));
    p[c2] = __builtin_convertvector(x, bf16x8);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bf16x2 pair = {p[c2][2 * e], p[c2][2 * e + 1]};
      ls = __builtin_amdgcn_fdot2_f32_bf16(pair, ones, ls, false);
    }
  }
  return ls;
}

// Scheduling hint for one half step: D/16 LDS reads and D/16 MFMAs of QK^T,
// D/16 transposed-read pairs and D/16 MFMAs of PV, and the weights of one block
// (about 50 VALU instructions). A few LDS reads go first, then each MFMA is
// followed by a slice of the VALU work and the next LDS reads, so the vector
// ALUs work while each MFMA runs.
template <int D>
__device__ __forceinline__ void interleave_half_step() {
  constexpr int kMfma = 2 * (D / 16);
  constexpr int kValu = 52 / kMfma + 1;
  __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);  // DS read
#pragma unroll
  for (int i = 0; i < kMfma; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);      // MFMA
    __builtin_amdgcn_sched_group_barrier(0x002, kValu, 0);  // VALU
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);      // DS read
  }
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
  float m_ref = -INFINITY;  // exponent reference (raw logit units) of this lane's query
  float l_run = 0.f;        // this lane's part of the running sum of weights
  const float lazy = exp2f(kLazyLog2);

  const int kbeg = row_ptr[frame];
  const int n_kept = row_ptr[frame + 1] - kbeg;
  const int tpf = (T + kBlockK - 1) / kBlockK;
  const int n_tiles = n_kept * tpf;

  if (n_tiles > 0) {
    Stage<D> kst, vst;
    // Prologue: K(0), V(0) and K(1) into LDS, scores of tile 0, then the loads of
    // K(2) and V(1), which step 0 stores.
    TileCursor kc, vc;
    kc.start(cols + kbeg, tpf, T);
    kst.load(Kh, kc.key0(), kc.nvalid(), tid);
    vst.load(Vh, kc.key0(), kc.nvalid(), tid);
    const int nv0 = kc.nvalid();
    kst.template store<Sh::kStrideK>(sK[0], tid);
    vst.template store<Sh::kStrideV>(sV[0], tid);
    kc.advance(n_kept);
    vc = kc;  // tile 1
    if (n_tiles > 1) {
      kst.load(Kh, kc.key0(), kc.nvalid(), tid);
      kst.template store<Sh::kStrideK>(sK[1], tid);
    }
    kc.advance(n_kept);  // tile 2
    __syncthreads();

    // Carried from one step to the next: the scores of the second block of tile
    // t (sa/sb) and the weights and their lane sum of its first block (pa/pb, la/lb).
    f32x16 sa, sb;
    bf16x8 pa[2], pb[2];
    float la = 0.f, lb = 0.f;
    if (wave_active) {
      f32x16 s0 = qk_block<D>(sK[0], qf, n, hf, 0);
      sa = qk_block<D>(sK[0], qf, n, hf, 1);
      if (nv0 < kBlockK) {
        mask_tail(s0, 0, hf, nv0);
        mask_tail(sa, 1, hf, nv0);
      }
      // The first tile sets the exponent reference.
      m_ref = pair_max(fmaxf(block_max(s0), block_max(sa)));
      la = block_weights(s0, c, m_ref * c, pa);
    }
    // Tiles that do not exist are loaded with an empty range (all zeros).
    kst.load(Kh, kc.key0(), n_tiles > 2 ? kc.nvalid() : 0, tid);
    vst.load(Vh, vc.key0(), n_tiles > 1 ? vc.nvalid() : 0, tid);
    kc.advance(n_kept);  // tile 3
    vc.advance(n_kept);  // tile 2
    int kt_next = tpf > 1 ? 1 : 0;  // index within its frame of tile t + 1
    // Step 0 overwrites K(0)'s buffer with K(2); every wave must be done reading it.
    __syncthreads();

    // Raise the exponent reference to cover block s, rescale what is accumulated
    // so far, and redo the block's weights.
    auto rescale = [&](const f32x16& s_blk, bf16x8(&p)[2], float& l) {
      const float m_new = fmaxf(m_ref, pair_max(block_max(s_blk)));
      const float alpha = fast_exp2((m_ref - m_new) * c);
      l_run *= alpha;
#pragma unroll
      for (int mb = 0; mb < Sh::kDBlocks; ++mb) o[mb] *= alpha;
      m_ref = m_new;
      l = block_weights(s_blk, c, m_ref * c, p);
    };

    // Step t, in two halves over 32-key blocks b = 2t, 2t+1:
    //   half 0: QK^T of block 2t+2 (tile t+1), weights of block 2t+1, PV of block 2t
    //   half 1: QK^T of block 2t+3 (tile t+1), weights of block 2t+2, PV of block 2t+1
    // The three parts of a half are independent, so their MFMAs and VALU work
    // interleave. Block b's weights are checked before its PV; a rescale at that
    // point multiplies exactly the blocks already accumulated. On the last step
    // the K buffer holds a stale tile: its scores and weights are never used.
    auto step = [&](int t, f32x16& s_in, bf16x8(&p_in)[2], float& l_in, f32x16& s_out,
                    bf16x8(&p_out)[2], float& l_out) {
      const bool have_next = t + 1 < n_tiles;
      // K(t+2) and V(t+1), loaded during the previous step, go to the buffers
      // that tile t and tile t-1 freed; then the loads of K(t+3) and V(t+2) start.
      kst.template store<Sh::kStrideK>(sK[t & 1], tid);
      vst.template store<Sh::kStrideV>(sV[(t + 1) & 1], tid);
      kst.load(Kh, kc.key0(), t + 3 < n_tiles ? kc.nvalid() : 0, tid);
      vst.load(Vh, vc.key0(), t + 2 < n_tiles ? vc.nvalid() : 0, tid);
      const uint16_t* kbuf = sK[(t + 1) & 1];
      const uint16_t* vbuf = sV[t & 1];
      const int nv_next = min(kBlockK, T - kt_next * kBlockK);
      if (wave_active) {
        f32x16 s2 = qk_block<D>(kbuf, qf, n, hf, 0);
        bf16x8 p1[2];
        float l1 = block_weights(s_in, c, m_ref * c, p1);
        pv_block<D>(vbuf, p_in, lane, 0, o);
        l_run += l_in;
        interleave_half_step<D>();
        if (__builtin_amdgcn_ballot_w64(l1 > lazy) != 0) rescale(s_in, p1, l1);
        if (have_next && nv_next < kBlockK) mask_tail(s2, 0, hf, nv_next);

        s_out = qk_block<D>(kbuf, qf, n, hf, 1);
        l_out = block_weights(s2, c, m_ref * c, p_out);
        pv_block<D>(vbuf, p1, lane, 1, o);
        l_run += l1;
        interleave_half_step<D>();
        if (have_next) {
          if (__builtin_amdgcn_ballot_w64(l_out > lazy) != 0) rescale(s2, p_out, l_out);
          if (nv_next < kBlockK) mask_tail(s_out, 1, hf, nv_next);
        }
      }
      kc.advance(n_kept);
      vc.advance(n_kept);
      if (++kt_next == tpf) kt_next = 0;
      __syncthreads();
    };

    int t = 0;
    for (; t + 1 < n_tiles; t += 2) {
      step(t, sa, pa, la, sb, pb, lb);
      step(t + 1, sb, pb, lb, sa, pa, la);
    }
    if (t < n_tiles) step(t, sa, pa, la, sb, pb, lb);
  }

  // Epilogue: normalise, round to bf16 (RNE), store 4 consecutive d per access.
  const float l_tot = pair_sum(l_run);
  if (qvalid) {
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
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
