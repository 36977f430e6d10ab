// gfx950 (MI355X, CDNA4) kernels for the tile-sparse 3D attention forward pass.
//
// What is computed (Sec. 3.3 of Efficient-vDiT): for every query token of latent
// frame i, softmax attention over the key tokens of the frames j that the
// frame mask keeps. Frames the mask drops are never read (App. B: empty blocks
// are skipped); the kernel walks a compact kept-frame list per query frame.
//
// Work decomposition
//   One workgroup = 4 waves = 256 query rows of one (batch, head, query frame);
//   each wave owns 64 rows as two 32-query column blocks (128 rows and one block
//   at d = 128, see fwd_q_blocks; at d = 64 a block at the end of a frame with at
//   most 32 valid rows per wave also runs one column block per wave, see
//   fwd_rows; at d = 64 and 96 a block with at most 32 valid rows in all runs on
//   two waves that split the keys of every tile, see fwd_tail_rows). Query blocks
//   are frame aligned, so every row of
//   a workgroup shares one kept list. With a text prefix (the MM-DiT form) the text
//   is one more segment, see Layout. Workgroup ids are
//   remapped so that each XCD (8 per MI355X, each with its own L2) receives a
//   contiguous run of (batch, head) problems, which keeps the K/V of the shared
//   global frames resident in that XCD's L2. Two workgroups share a CU, so each
//   SIMD runs two waves: while one forms softmax weights on the vector ALUs the
//   other keeps the matrix cores busy.
//
// Matrix-core layout (v_mfma_f32_32x32x16_bf16, wave64)
//   A (32 x 16): lane l holds row l%32, k = 8*(l/32) .. +7
//   B (16 x 32): lane l holds col l%32, k = 8*(l/32) .. +7
//   C (32 x 32): lane l holds col l%32, rows 8*i + 4*(l/32) + j at index 4*i + j
//   The kernel computes S^T = K * Q^T (A = K rows from LDS, B = the wave's queries
//   held in registers), so each lane owns one query per column block and 16 of
//   every 32 keys. The probabilities P^T then sit exactly where the B operand of
//   O^T += V^T * P^T expects them, with the contraction index k of chunk ch mapped
//   to keys 16ch + 4h + (0..3) and 16ch + 8 + 4h + (0..3) for lane half h. Every
//   K and V^T fragment read from LDS feeds two MFMAs (both column blocks), which
//   halves the LDS read traffic per matrix instruction.
//   The V^T operand is read from the untransposed V tile with the LDS transpose
//   load ds_read_b64_tr_b16: inside each 16-lane group, lane i receives element
//   i%4 of the 8-byte rows read by lanes 4k + i/4 (k = 0..3), so when lane j reads
//   V[key0 + j/4][d0 + 4(j%4) .. +3], lane i gets V[key0 .. key0+3][d0 + i].
//
// Tiles (64 keys) move from global memory straight into LDS with buffer loads
// that write LDS (no register staging). K and V each have two LDS buffers: while
// tile t is consumed, tile t+1 lands in the other pair; one barrier per tile.
//
// Online softmax (fp32, base 2): weights are exp2(c * (s - m_ref)) with
// c = |scale| * log2(e) and m_ref an exponent reference per query that only
// moves when needed. Weights are formed directly; if any lane's sum of weights
// in a 32-key block exceeds 2^kLazyLog2 (so some weight may have grown past it;
// at the first block m_ref = -inf makes them infinite or NaN), the block is redone with
// m_ref raised to the running max and O^T and l rescaled. Weights up to
// 2^kLazyLog2 are as exact in fp32 and bf16 as weights up to 1, so the result is
// the same softmax; only the reference of the exponentials moves less often. The
// row sum l is accumulated from the bf16-rounded weights that also feed the PV
// product, per lane (its 16 of every 32 keys) and summed over the two lane
// halves once, in the epilogue.
#include <hip/hip_runtime.h>

#include <float.h>

#include <algorithm>
#include <type_traits>
#include <stdint.h>

#include "launch.h"
#include "tile_common.h"
#include "unit_order.h"

namespace ta {
namespace {

constexpr int kWaves = kThreads / 64;
constexpr float kLazyLog2 = 10.f;
// 32-query column blocks per wave: two (64 rows, every LDS fragment feeds two MFMAs)
// where they fit 256 VGPRs, one at d = 128 (two spilled some 70 VGPRs inside the
// tile loop and ran at half the rate).
template <int D>
constexpr int fwd_q_blocks() { return D == 128 ? 1 : 2; }
template <int D>
constexpr int fwd_rows_per_wg() { return kWaves * 32 * fwd_q_blocks<D>(); }

template <int D>
struct Shape {
  static constexpr int kChunks = D / 16;   // 16-wide slices of the QK^T contraction
  static constexpr int kDBlocks = D / 32;  // 32-row blocks of O^T
  static constexpr int kPieces = D / 8;    // 16-byte pieces per K/V row
  static constexpr int kTileElems = kBlockK * D;
  // 16-byte direct loads per wave to fill one K or V tile (one load = 64 pieces).
  static constexpr int kLoadsPerWave = kBlockK * kPieces / 64 / kWaves;
  static_assert(kBlockK * kPieces == 64 * kWaves * kLoadsPerWave, "whole loads per wave");
};

// LDS tile layouts. A tile is kBlockK rows (keys) of D bf16, stored as rows of
// kPieces 16-byte pieces with the pieces of each row permuted by an XOR, so that
// the MFMA operand reads hit distinct banks:
//   K (read 16 bytes per lane, 16 consecutive rows per access): piece p of row r
//     sits at p ^ ksw(r), which spreads those 16 rows over all 64 banks;
//   V (read 8 bytes per lane by the transpose load, 4 consecutive rows x 64 bytes
//     per access): the 64-byte quads of row r are permuted by vsw(r), which puts
//     those 4 rows in 4 different 64-byte bank groups.
// Both XORs keep every aligned group of four pieces together, so one direct load
// (64 lanes x 16 bytes into 1 KB of LDS) reads 1 KB of contiguous global memory.
template <int D>
__device__ __forceinline__ int ksw(int r) {
  if constexpr (D == 64) return (r >> 1) & 7;
  else if constexpr (D == 96) return (r >> 2) & 3;
  else return r & 15;
}
template <int D>
__device__ __forceinline__ int vsw(int r) {
  if constexpr (D == 64) return ((r >> 1) & 1) << 2;
  else if constexpr (D == 96) return 0;
  else return (r & 3) << 2;
}
// Element offset in LDS of piece p (8 bf16) of row r.
template <int D>
__device__ __forceinline__ int k_slot(int r, int p) { return (r * (D / 8) + (p ^ ksw<D>(r))) * 8; }
template <int D>
__device__ __forceinline__ int v_slot(int r, int p) { return (r * (D / 8) + (p ^ vsw<D>(r))) * 8; }

// Direct global -> LDS loads of one 64-key K or V tile (kBlockK * D contiguous bf16
// in global memory). Load j of wave w fills LDS pieces [64 i, 64 i + 64) with
// i = w + kWaves * j; lane L fills piece 64 i + L, which the layout maps back to
// row r and source piece p. The source byte offsets depend only on the lane, so
// they are computed once.
template <int D, bool IS_K>
struct TileLoader {
  int off[Shape<D>::kLoadsPerWave];  // source byte offset within the tile, per load
  __device__ __forceinline__ void init(int wave, int lane) {
#pragma unroll
    for (int j = 0; j < Shape<D>::kLoadsPerWave; ++j) {
      const int q = 64 * (wave + kWaves * j) + lane;
      const int r = q / Shape<D>::kPieces, ps = q % Shape<D>::kPieces;
      const int p = ps ^ (IS_K ? ksw<D>(r) : vsw<D>(r));
      off[j] = (r * D + 8 * p) * 2;
    }
  }
  // Rows past nvalid read as zeros (buffer range check).
  __device__ __forceinline__ void load(const uint16_t* Xh, size_t key0, int nvalid,
                                       const uint16_t* lds, int wave) const {
    const i32x4 rs = buffer_words(Xh + key0 * D, (uint32_t)(nvalid * D * 2));
    const uint32_t base = lds_addr(lds);
#pragma unroll
    for (int j = 0; j < Shape<D>::kLoadsPerWave; ++j)
      load_to_lds(rs, __builtin_amdgcn_readfirstlane(base + 1024u * (uint32_t)(wave + kWaves * j)),
                  off[j]);
  }
};

// Per-lane LDS element offsets of this lane's K fragment pieces for 32-key block
// 0 of a tile (row n of the block, piece 2 cc + h of each 16-wide chunk cc); the
// swizzle of a row depends only on n, so block kb adds kb * 32 * D.
template <int D>
struct KAddr {
  int at[D / 16];
  __device__ __forceinline__ void init(int n, int hf) {
#pragma unroll
    for (int cc = 0; cc < D / 16; ++cc) at[cc] = k_slot<D>(n, 2 * cc + hf);
  }
};

// Per-lane LDS element offsets of this lane's transposed V reads for key chunk 0
// of a tile, one per 32-row d-block: lane l (group g = l/16, j = l%16) reads
// V[4(g/2) + j/4][32mb + 16(g%2) + 4(j%4) .. +3]. Chunk ch adds 16 ch * D and the
// second read (keys + 8) adds 8 * D: the swizzle of a row depends only on its
// low two bits, which those steps do not change.
template <int D>
struct VAddr {
  int at[D / 32];
  __device__ __forceinline__ void init(int lane) {
    const int g = lane >> 4, j = lane & 15;
    const int r = 4 * (g >> 1) + (j >> 2);
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb)
      at[mb] = v_slot<D>(r, 4 * mb + 2 * (g & 1) + ((j >> 1) & 1)) + 4 * (j & 1);
  }
};

// S^T of 32-key block kb of a K tile for both 32-query column blocks of the wave
// (32 keys x 32 queries each), raw logits. Each K fragment feeds two MFMAs.
template <int D, int QB>
__device__ __forceinline__ void qk_block(const uint16_t* sK, const bf16x8 (&qf)[QB][D / 16],
                                         const KAddr<D>& ka, int kb, f32x16 (&s)[QB]) {
  const uint16_t* base = sK + kb * 32 * D;
  const bf16x8 a0 = as_bf16x8(load16(base + ka.at[0]));
#pragma unroll
  for (int qs = 0; qs < QB; ++qs) s[qs] = mfma32(a0, qf[qs][0], f32x16{});
#pragma unroll
  for (int cc = 1; cc < D / 16; ++cc) {
    const bf16x8 a = as_bf16x8(load16(base + ka.at[cc]));
#pragma unroll
    for (int qs = 0; qs < QB; ++qs) s[qs] = mfma32(a, qf[qs][cc], s[qs]);
  }
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
// chunk ch from the V tile: lane i of each 16-lane group receives
// V[key0 .. key0+3][d0 + i] from each of the two transposed reads (keys and
// keys + 8).
template <int D>
__device__ __forceinline__ bf16x8 vt_frag(const uint16_t* sV, const VAddr<D>& va, int mb, int ch) {
  const uint16_t* p = sV + 16 * ch * D + va.at[mb];
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 8 * D));
  const u32x2 a = __builtin_bit_cast(u32x2, lo), b = __builtin_bit_cast(u32x2, hi);
  return as_bf16x8(u32x4{a[0], a[1], b[0], b[1]});
}

// O^T (d x 32 queries, both column blocks) += V^T * P^T over 32-key block kb (key
// chunks 2kb, 2kb+1). Each V^T fragment feeds two MFMAs.
template <int D, int QB>
__device__ __forceinline__ void pv_block(const uint16_t* sV, const bf16x8 (&p)[QB][2],
                                         const VAddr<D>& va, int kb, f32x16 (&o)[QB][D / 32]) {
#pragma unroll
  for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb) {
      const bf16x8 a = vt_frag<D>(sV, va, mb, 2 * kb + c2);
#pragma unroll
      for (int qs = 0; qs < QB; ++qs) o[qs][mb] = mfma32(a, p[qs][c2], o[qs][mb]);
    }
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

// The weights of keys 2e and 2e+1 of chunk c2 of a 32-key block for one column
// block, exactly as block_weights forms them: one packed dword of the B operand,
// and their bf16 values added to this lane's sum.
__device__ __forceinline__ void pair_weights(const f32x16& s, int c2, int e, float c, float mc,
                                             u32x4& pw, float& ls) {
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  const f32x2 x = {fast_exp2(__builtin_fmaf(s[8 * c2 + 2 * e], c, -mc)),
                   fast_exp2(__builtin_fmaf(s[8 * c2 + 2 * e + 1], c, -mc))};
  const bf16x2 y = __builtin_convertvector(x, bf16x2);
  pw[e] = __builtin_bit_cast(uint32_t, y);
  ls = __builtin_amdgcn_fdot2_f32_bf16(y, ones, ls, false);
}

// fn(integral_constant<int, i>) for i = 0 .. N-1, in order.
template <int N, int I = 0, typename Fn>
__device__ __forceinline__ void static_for(Fn&& fn) {
  if constexpr (I < N) {
    fn(std::integral_constant<int, I>{});
    static_for<N, I + 1>(static_cast<Fn&&>(fn));
  }
}

// One workgroup's work item, decoded: the (batch, head) slabs, the query segment
// and its query block, and the kept list.
struct FwdItem {
  const uint16_t* Qh;
  const uint16_t* Kh;
  const uint16_t* Vh;
  uint16_t* Oh;
  const int32_t* cols;
  size_t head_rows;
  uint32_t b, bh, B;
  int frame, kbeg, n_kept, slot, qb, seg0, seg_len;
  // Tiles of the kept list this workgroup takes: [t0, t0 + nt), nt < 0 for all of
  // them; a part of the list (part >= 0) writes its rows to block `part` of ws_parts.
  int t0, nt, part;
};

// Epilogue of a wave's QB column blocks, whose first row (within the segment) is
// row0: normalise; a whole frame rounds to bf16 (RNE) into out, a piece of a split
// frame stores O/l in fp32 and its base-2 log-sum-exp log2(sum_t 2^(c s_t)) =
// c m_ref + log2(l) for the merge, and a part of the kept tiles (part >= 0) stores
// the same to its own slot. 4 consecutive d per access. The lane's rows are derived
// from a lane id read here, so that nothing lane-dependent from before the tile loop
// has to stay live across it.
template <int D, bool PREFIX, int QB>
__device__ __forceinline__ void store_rows(const FwdItem& it, int row0, int part,
                                           const f32x16 (&o)[QB][Shape<D>::kDBlocks], const float (&m_ref)[QB],
                                           const float (&l_run)[QB], float c, int T, int P, float* __restrict__ lse,
                                           float* __restrict__ ws_o, float* __restrict__ ws_lse,
                                           float* __restrict__ ws_parts) {
  using Sh = Shape<D>;
  constexpr int kBlockQ = fwd_rows_per_wg<D>();
  const int seg0 = it.seg0, seg_len = it.seg_len, slot = it.slot, qb = it.qb;
  // The row offsets below are formed here, after the tile loop: values derived from
  // them are not worth a scalar register across the loop.
  asm volatile("" : "+s"(T), "+s"(P));
  int lane_e;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lane_e));
  const int hf_e = lane_e >> 5;
  const int qrow0_e = row0 + (lane_e & 31);
#pragma unroll
  for (int qs = 0; qs < QB; ++qs) {
    const float l_tot = pair_sum(l_run[qs]);
    const int qrow = qrow0_e + 32 * qs;
    if (qrow < seg_len) {
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      if (slot < 0 && part < 0) {
        uint16_t* op = it.Oh + ((size_t)seg0 + qrow) * D;
#pragma unroll
        for (int mb = 0; mb < Sh::kDBlocks; ++mb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            f32x4 x = {o[qs][mb][4 * i + 0] * inv, o[qs][mb][4 * i + 1] * inv,
                       o[qs][mb][4 * i + 2] * inv, o[qs][mb][4 * i + 3] * inv};
            const bf16x4 y = __builtin_convertvector(x, bf16x4);
            *reinterpret_cast<u32x2*>(op + 32 * mb + 8 * i + 4 * hf_e) = __builtin_bit_cast(u32x2, y);
          }
        if (lse && hf_e == 0)
          lse[(size_t)it.bh * it.head_rows + seg0 + qrow] =
              l_tot > 0.f ? (m_ref[qs] * c + __builtin_amdgcn_logf(l_tot)) * 0.69314718055994531f
                          : -INFINITY;
      } else {
        // A part of the kept tiles (part >= 0) goes to its own slot of kBlockQ rows of
        // D + 4 floats (O/l, then the log-sum-exp), a piece of a split frame (slot >= 0)
        // to the frame's partial rows.
        const int slot_rows = PREFIX ? max(T, P) : T;  // rows per (slot, batch entry)
        const size_t prow = part >= 0 ? (size_t)part * kBlockQ + (qrow - qb * kBlockQ)
                                    : ((size_t)slot * it.B + it.b) * slot_rows + qrow;
        float* op = part >= 0 ? ws_parts + prow * (D + 4) : ws_o + prow * D;
#pragma unroll
        for (int mb = 0; mb < Sh::kDBlocks; ++mb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const f32x4 x = {o[qs][mb][4 * i + 0] * inv, o[qs][mb][4 * i + 1] * inv,
                             o[qs][mb][4 * i + 2] * inv, o[qs][mb][4 * i + 3] * inv};
            *reinterpret_cast<f32x4*>(op + 32 * mb + 8 * i + 4 * hf_e) = x;
          }
        if (hf_e == 0) *(part >= 0 ? op + D : ws_lse + prow) = m_ref[qs] * c + __builtin_amdgcn_logf(l_tot);
      }
    }
  }
}

// The rows of one workgroup with QB 32-query column blocks per wave. The grid's
// query blocks hold fwd_rows_per_wg<D>() rows whatever QB is: at d = 64 a block at the
// end of a segment with at most 32 valid rows per wave runs with QB = 1, so no wave
// computes a column block that lies wholly past the segment end.
template <int D, bool PREFIX, int QB, bool TABLE>
__device__ __forceinline__ void fwd_rows(int wave, const FwdItem& it, const Layout<PREFIX>& lay,
                                         uint16_t (&sK)[2][Shape<D>::kTileElems],
                                         uint16_t (&sV)[2][Shape<D>::kTileElems],
                                         float* __restrict__ ws_o, float* __restrict__ ws_lse,
                                         float* __restrict__ lse, float* __restrict__ ws_parts, float c,
                                         uint32_t qflip, uint32_t qmask) {
  using Sh = Shape<D>;
  constexpr int kWaveQ = 32 * QB;
  constexpr int kBlockQ = fwd_rows_per_wg<D>();
  const uint16_t* Qh = it.Qh;
  const uint16_t* Kh = it.Kh;
  const uint16_t* Vh = it.Vh;
  const int32_t* cols = it.cols;
  const int kbeg = it.kbeg, n_kept = it.n_kept, qb = it.qb;
  const int part = TABLE ? it.part : -1;
  const int seg0 = it.seg0, seg_len = it.seg_len;
  [[maybe_unused]] const int F = lay.F, T = lay.T, P = lay.P;

  // The lane id is read here (an asm statement the compiler cannot hoist), so nothing
  // lane-dependent is held in vector registers across the caller's work loop; the
  // wave index comes in as a scalar.
  int lane;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lane));
  const int n = lane & 31, hf = lane >> 5;

  // This lane's two query rows (within the frame), one per 32-query column block,
  // and their Q^T B-operand slices.
  const int qrow0 = qb * kBlockQ + wave * kWaveQ + n;
  // Waves whose rows all lie past the frame end only help load tiles.
  const bool wave_active = qb * kBlockQ + wave * kWaveQ < seg_len;
  bf16x8 qf[QB][Sh::kChunks];
#pragma unroll
  for (int qs = 0; qs < QB; ++qs) {
    const int qrow = qrow0 + 32 * qs;
    const uint16_t* qp = Qh + ((size_t)seg0 + qrow) * D + 8 * hf;
#pragma unroll
    for (int cc = 0; cc < Sh::kChunks; ++cc) {
      u32x4 x = {0u, 0u, 0u, 0u};
      if (qrow < seg_len) x = (load16(qp + 16 * cc) & qmask) ^ qflip;
      qf[qs][cc] = as_bf16x8(x);
    }
  }

  f32x16 o[QB][Sh::kDBlocks];
#pragma unroll
  for (int qs = 0; qs < QB; ++qs)
#pragma unroll
    for (int mb = 0; mb < Sh::kDBlocks; ++mb) o[qs][mb] = f32x16{};
  // Per column block: exponent reference (raw logit units) of this lane's query
  // and this lane's part of the running sum of weights.
  float m_ref[QB], l_run[QB];
#pragma unroll
  for (int qs = 0; qs < QB; ++qs) {
    m_ref[qs] = -INFINITY;
    l_run[qs] = 0.f;
  }
  const float lazy = exp2f(kLazyLog2);

  const int tpf = (T + kBlockK - 1) / kBlockK;
  int n_tiles = n_kept * tpf;
  if constexpr (PREFIX) {
    // the text segment (index F) sorts last in a kept list
    if (n_kept > 0 && cols[kbeg + n_kept - 1] == F) n_tiles += (P + kBlockK - 1) / kBlockK - tpf;
  }
  if constexpr (TABLE) {
    if (it.nt >= 0) n_tiles = it.nt;  // a part of the kept tiles, from tile it.t0
  }

  if (n_tiles > 0) {
    TileLoader<D, true> kl;
    TileLoader<D, false> vl;
    kl.init(wave, lane);
    vl.init(wave, lane);
    KAddr<D> ka;
    VAddr<D> va;
    ka.init(n, hf);
    va.init(lane);
    SegmentCursor<PREFIX> cur, nxt;  // tile t (being consumed) and tile t+1 (being loaded)
    cur.start(cols + kbeg, lay);
    if constexpr (TABLE) {
      if (it.t0 > 0) cur.skip(it.t0, n_kept);
    }
    kl.load(Kh, cur.key0(), cur.nvalid(), sK[0], wave);
    vl.load(Vh, cur.key0(), cur.nvalid(), sV[0], wave);
    nxt = cur;
    nxt.advance(n_kept);
    wait_tile_loads();
    __syncthreads();

    // The weights of a block are used only once every lane's sum of them is at
    // most 2^kLazyLog2; otherwise (written so that NaN also qualifies: at the first
    // block m_ref = -inf turns masked keys into NaN weights) the references are
    // raised to cover the block, what is accumulated so far is rescaled, and the
    // block's weights are redone. Then the block's sums join the running sums.
    auto check_block = [&](const f32x16(&s)[QB], bf16x8(&p)[QB][2], float(&ls)[QB]) {
      bool small = true;
#pragma unroll
      for (int qs = 0; qs < QB; ++qs) small = small && ls[qs] <= lazy;
      if (__builtin_amdgcn_ballot_w64(!small) != 0) {
#pragma unroll
        for (int qs = 0; qs < QB; ++qs) {
          const float m_new = fmaxf(m_ref[qs], pair_max(block_max(s[qs])));
          const float alpha = fast_exp2((m_ref[qs] - m_new) * c);
          l_run[qs] *= alpha;
#pragma unroll
          for (int mb = 0; mb < Sh::kDBlocks; ++mb) o[qs][mb] *= alpha;
          m_ref[qs] = m_new;
          ls[qs] = block_weights(s[qs], c, m_new * c, p[qs]);
        }
      }
#pragma unroll
      for (int qs = 0; qs < QB; ++qs) l_run[qs] += ls[qs];
    };

    // One tile; the buffer index is a compile-time constant (the loop below runs tiles
    // in pairs), so every LDS address is a per-lane base plus an immediate offset.
    auto tile_step = [&](auto bufc, int t) {
      constexpr int buf = decltype(bufc)::value;
      // Tile t+1 lands in the buffers tile t-1 freed (all waves passed the last
      // barrier) while tile t is consumed.
      if (t + 1 < n_tiles) {
        kl.load(Kh, nxt.key0(), nxt.nvalid(), sK[buf ^ 1], wave);
        vl.load(Vh, nxt.key0(), nxt.nvalid(), sV[buf ^ 1], wave);
      }
      const int nvalid = cur.nvalid();
      if (wave_active) {
        // Within the tile: QK^T of block 1 runs on the matrix cores while the
        // weights of block 0 form on the vector ALUs, then PV of block 0 while the
        // weights of block 1 form, then PV of block 1.
        f32x16 s0[QB], s1[QB];
        bf16x8 p0[QB][2], p1[QB][2];
        float l0[QB], l1[QB];
        qk_block<D, QB>(sK[buf], qf, ka, 0, s0);
        if (nvalid < kBlockK) {
#pragma unroll
          for (int qs = 0; qs < QB; ++qs) mask_tail(s0[qs], 0, hf, nvalid);
        }
        // Two regions: QK^T of block 1 with the weights of block 0, then PV of block 0
        // with the weights of block 1. Each holds QB * D/16 MFMAs and 16 QB weights.
        constexpr int kMfma = QB * (D / 16);
        if constexpr (QB == 2) {
          // Written as packets of one MFMA and an even share of the weight pairs, with
          // a scheduling fence after each, so the vector work issues while the matrix
          // core runs (about 2% faster at d = 64 and 96 than a scheduling hint per
          // region). Operand fragments are read from LDS two packets before their
          // first use, into three rotating registers, and the last packets of a region
          // already read the first two V^T fragments of the next PV region (1% more).
          constexpr int kPairs = QB * 8;
          constexpr int kMb = D / 32;  // V^T fragment f of a block: chunk f / kMb, d-block f % kMb
          float mc[QB];
          u32x4 pw[QB][2];
          bf16x8 vn[2];  // the first two V^T fragments of the next PV region
          auto weights_share = [&](auto ic, const f32x16(&sb)[QB], float(&ls)[QB]) {
            constexpr int i = decltype(ic)::value;
#pragma unroll
            for (int j = i * kPairs / kMfma; j < (i + 1) * kPairs / kMfma; ++j)
              pair_weights(sb[j / 8], (j / 4) % 2, j % 4, c, mc[j / 8], pw[j / 8][(j / 4) % 2],
                           ls[j / 8]);
          };
          auto start_weights = [&](float(&ls)[QB]) {
#pragma unroll
            for (int qs = 0; qs < QB; ++qs) {
              mc[qs] = m_ref[qs] * c;
              ls[qs] = 0.f;
            }
          };
          auto finish_weights = [&](bf16x8(&p)[QB][2]) {
#pragma unroll
            for (int qs = 0; qs < QB; ++qs)
#pragma unroll
              for (int c2 = 0; c2 < 2; ++c2) p[qs][c2] = __builtin_bit_cast(bf16x8, pw[qs][c2]);
          };
          // O^T += V^T * P^T over block kb, one packet per MFMA; extra(ic) adds the
          // packet's vector work. Block 0's packets read block 1's first fragments.
          auto pv_packets = [&](auto kbc, const bf16x8(&p)[QB][2], auto&& extra) {
            constexpr int kb = decltype(kbc)::value;
            bf16x8 vf[3];
            vf[0] = vn[0];
            vf[1] = vn[1];
            static_for<kMfma>([&](auto ic) {
              constexpr int i = decltype(ic)::value, f = i / QB, qs = i % QB, g = f + 2 - 2 * kMb;
              if constexpr (qs == 0 && g < 0)
                vf[(f + 2) % 3] = vt_frag<D>(sV[buf], va, (f + 2) % kMb, 2 * kb + (f + 2) / kMb);
              if constexpr (kb == 0 && qs == 0 && g >= 0) vn[g] = vt_frag<D>(sV[buf], va, g % kMb, 2 + g / kMb);
              o[qs][f % kMb] = mfma32(vf[f % 3], p[qs][f / kMb], o[qs][f % kMb]);
              extra(ic);
              __builtin_amdgcn_sched_barrier(0);
            });
          };

          start_weights(l0);
          {
            const uint16_t* kb1 = sK[buf] + 32 * D;
            bf16x8 kf[3];
            kf[0] = as_bf16x8(load16(kb1 + ka.at[0]));
            kf[1] = as_bf16x8(load16(kb1 + ka.at[1]));
            __builtin_amdgcn_sched_barrier(0);
            static_for<kMfma>([&](auto ic) {
              constexpr int i = decltype(ic)::value, cc = i / QB, qs = i % QB, g = cc + 2 - D / 16;
              if constexpr (qs == 0 && g < 0) kf[(cc + 2) % 3] = as_bf16x8(load16(kb1 + ka.at[cc + 2]));
              if constexpr (qs == 0 && g >= 0) vn[g] = vt_frag<D>(sV[buf], va, g % kMb, g / kMb);
              s1[qs] = mfma32(kf[cc % 3], qf[qs][cc], cc == 0 ? f32x16{} : s1[qs]);
              weights_share(ic, s0, l0);
              __builtin_amdgcn_sched_barrier(0);
            });
          }
          finish_weights(p0);
          check_block(s0, p0, l0);
          if (nvalid < kBlockK) {
#pragma unroll
            for (int qs = 0; qs < QB; ++qs) mask_tail(s1[qs], 1, hf, nvalid);
          }
          start_weights(l1);
          pv_packets(std::integral_constant<int, 0>{}, p0, [&](auto ic) { weights_share(ic, s1, l1); });
          finish_weights(p1);
          check_block(s1, p1, l1);
          pv_packets(std::integral_constant<int, 1>{}, p1, [](auto) {});
        } else {
          // One column block (d = 128): the regions are fenced and the vector work is
          // spread evenly between the MFMAs by a scheduling hint (about 48 vector
          // instructions per block: fma, exp, half a conversion, half a dot2 per
          // element).
          constexpr int kValuPerMfma = 768 / D;
          __builtin_amdgcn_sched_barrier(0);
          qk_block<D, QB>(sK[buf], qf, ka, 1, s1);
#pragma unroll
          for (int qs = 0; qs < QB; ++qs) l0[qs] = block_weights(s0[qs], c, m_ref[qs] * c, p0[qs]);
          spread_valu_over_mfma<kMfma, kValuPerMfma>();
          check_block(s0, p0, l0);
          if (nvalid < kBlockK) {
#pragma unroll
            for (int qs = 0; qs < QB; ++qs) mask_tail(s1[qs], 1, hf, nvalid);
          }
          __builtin_amdgcn_sched_barrier(0);
          pv_block<D, QB>(sV[buf], p0, va, 0, o);
#pragma unroll
          for (int qs = 0; qs < QB; ++qs) l1[qs] = block_weights(s1[qs], c, m_ref[qs] * c, p1[qs]);
          spread_valu_over_mfma<kMfma, kValuPerMfma>();
          check_block(s1, p1, l1);
          __builtin_amdgcn_sched_barrier(0);
          pv_block<D, QB>(sV[buf], p1, va, 1, o);
        }
      }
      cur = nxt;
      nxt.advance(n_kept);
      wait_tile_loads();
      __syncthreads();
    };
    for (int t = 0; t < n_tiles; t += 2) {
      tile_step(std::integral_constant<int, 0>{}, t);
      if (t + 1 < n_tiles) tile_step(std::integral_constant<int, 1>{}, t + 1);
    }
  }

  store_rows<D, PREFIX, QB>(it, qb * kBlockQ + wave * kWaveQ, part, o, m_ref, l_run, c, T, P, lse, ws_o,
                            ws_lse, ws_parts);
}

// A query block with at most 32 valid rows (the short last block of a segment, such
// as the 16 rows left at T = 3600): one 32-query column block, shared by waves 0 and
// 1, which take the two 32-key halves of every tile; waves 2 and 3 only load tiles.
// Wave 1's softmax state (reference, sum, O^T) then joins wave 0's through LDS and
// wave 0 stores the rows. Each tile costs an active wave a quarter of the matrix and
// vector work of a full block's wave, so the block frees its workgroup slot early
// instead of holding it for one wave's whole pass over the tiles.
template <int D, bool PREFIX, bool TABLE>
__device__ __forceinline__ void fwd_tail_rows(int wave, const FwdItem& it, const Layout<PREFIX>& lay,
                                              uint16_t (&sK)[2][Shape<D>::kTileElems],
                                              uint16_t (&sV)[2][Shape<D>::kTileElems],
                                              float* __restrict__ ws_o, float* __restrict__ ws_lse,
                                              float* __restrict__ lse, float* __restrict__ ws_parts, float c,
                                              uint32_t qflip, uint32_t qmask) {
  using Sh = Shape<D>;
  constexpr int kBlockQ = fwd_rows_per_wg<D>();
  const int32_t* cols = it.cols;
  const int kbeg = it.kbeg, n_kept = it.n_kept, qb = it.qb;
  const int part = TABLE ? it.part : -1;
  const int seg0 = it.seg0, seg_len = it.seg_len;
  [[maybe_unused]] const int F = lay.F, T = lay.T, P = lay.P;

  int lane;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lane));
  const int n = lane & 31, hf = lane >> 5;
  const bool wave_active = wave < 2;  // wave w takes keys 32 w .. 32 w + 31 of every tile

  bf16x8 qf[1][Sh::kChunks];
  {
    const int qrow = qb * kBlockQ + n;
    const uint16_t* qp = it.Qh + ((size_t)seg0 + qrow) * D + 8 * hf;
#pragma unroll
    for (int cc = 0; cc < Sh::kChunks; ++cc) {
      u32x4 x = {0u, 0u, 0u, 0u};
      if (qrow < seg_len) x = (load16(qp + 16 * cc) & qmask) ^ qflip;
      qf[0][cc] = as_bf16x8(x);
    }
  }
  f32x16 o[1][Sh::kDBlocks];
#pragma unroll
  for (int mb = 0; mb < Sh::kDBlocks; ++mb) o[0][mb] = f32x16{};
  float m_ref[1] = {-INFINITY}, l_run[1] = {0.f};
  const float lazy = exp2f(kLazyLog2);

  const int tpf = (T + kBlockK - 1) / kBlockK;
  int n_tiles = n_kept * tpf;
  if constexpr (PREFIX) {
    if (n_kept > 0 && cols[kbeg + n_kept - 1] == F) n_tiles += (P + kBlockK - 1) / kBlockK - tpf;
  }
  if constexpr (TABLE) {
    if (it.nt >= 0) n_tiles = it.nt;
  }

  if (n_tiles > 0) {
    TileLoader<D, true> kl;
    TileLoader<D, false> vl;
    kl.init(wave, lane);
    vl.init(wave, lane);
    KAddr<D> ka;
    VAddr<D> va;
    ka.init(n, hf);
    va.init(lane);
    SegmentCursor<PREFIX> cur, nxt;
    cur.start(cols + kbeg, lay);
    if constexpr (TABLE) {
      if (it.t0 > 0) cur.skip(it.t0, n_kept);
    }
    kl.load(it.Kh, cur.key0(), cur.nvalid(), sK[0], wave);
    vl.load(it.Vh, cur.key0(), cur.nvalid(), sV[0], wave);
    nxt = cur;
    nxt.advance(n_kept);
    wait_tile_loads();
    __syncthreads();

    auto tile_step = [&](auto bufc, int t) {
      constexpr int buf = decltype(bufc)::value;
      if (t + 1 < n_tiles) {
        kl.load(it.Kh, nxt.key0(), nxt.nvalid(), sK[buf ^ 1], wave);
        vl.load(it.Vh, nxt.key0(), nxt.nvalid(), sV[buf ^ 1], wave);
      }
      const int nvalid = cur.nvalid();
      // A half with no valid key (the second half of a frame's last tile of at most
      // 32 keys) is skipped: its weights would be NaN while the reference is -inf.
      if (wave_active && 32 * wave < nvalid) {
        f32x16 s[1];
        bf16x8 p[1][2];
        qk_block<D, 1>(sK[buf], qf, ka, wave, s);
        if (nvalid < 32 * (wave + 1)) mask_tail(s[0], wave, hf, nvalid);
        float ls = block_weights(s[0], c, m_ref[0] * c, p[0]);
        // As in the full blocks: the weights are kept when every lane's sum is at
        // most 2^kLazyLog2, else the reference is raised and the block redone.
        if (__builtin_amdgcn_ballot_w64(!(ls <= lazy)) != 0) {
          const float m_new = fmaxf(m_ref[0], pair_max(block_max(s[0])));
          const float alpha = fast_exp2((m_ref[0] - m_new) * c);
          l_run[0] *= alpha;
#pragma unroll
          for (int mb = 0; mb < Sh::kDBlocks; ++mb) o[0][mb] *= alpha;
          m_ref[0] = m_new;
          ls = block_weights(s[0], c, m_new * c, p[0]);
        }
        l_run[0] += ls;
        pv_block<D, 1>(sV[buf], p, va, wave, o);
      }
      cur = nxt;
      nxt.advance(n_kept);
      wait_tile_loads();
      __syncthreads();
    };
    for (int t = 0; t < n_tiles; t += 2) {
      tile_step(std::integral_constant<int, 0>{}, t);
      if (t + 1 < n_tiles) tile_step(std::integral_constant<int, 1>{}, t + 1);
    }

    // Every wave has passed the last tile's barrier and no load is in flight, so the
    // K buffers hold wave 1's state: value i of lane l at float i * 64 + l.
    float* xs = reinterpret_cast<float*>(&sK[0][0]);
    if (wave == 1) {
      xs[lane] = m_ref[0];
      xs[64 + lane] = l_run[0];
#pragma unroll
      for (int mb = 0; mb < Sh::kDBlocks; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) xs[(2 + 16 * mb + r) * 64 + lane] = o[0][mb][r];
    }
    __syncthreads();
    if (wave == 0) {
      // Wave 0 saw the first half of every tile, which always holds a valid key, so
      // its reference is finite; wave 1's is -inf if it saw none (weight 0 below).
      const float m1 = xs[lane];
      const float m_new = fmaxf(m_ref[0], m1);
      const float a0 = fast_exp2((m_ref[0] - m_new) * c), a1 = fast_exp2((m1 - m_new) * c);
      l_run[0] = l_run[0] * a0 + xs[64 + lane] * a1;
#pragma unroll
      for (int mb = 0; mb < Sh::kDBlocks; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[0][mb][r] = o[0][mb][r] * a0 + xs[(2 + 16 * mb + r) * 64 + lane] * a1;
      m_ref[0] = m_new;
    }
  }
  if (wave == 0)
    store_rows<D, PREFIX, 1>(it, qb * kBlockQ, part, o, m_ref, l_run, c, T, P, lse, ws_o, ws_lse, ws_parts);
}

// One unit of work. Logical unit u = (batch entry b, item i, query block qb), qb
// fastest, covers the item's kept tiles for kBlockQ query rows. XCD x (the workgroups
// with blockIdx % 8 == x; each XCD has its own L2) owns the positions 0 .. n_x - 1 of
// its queue: positions below n_dp_x are the units start_x + pos, run whole; the
// n_tab_x after them are table entries {u, first tile, tiles, partial slot}: a part of
// a unit that would otherwise make a ragged last round of whole units (slot >= 0), or
// a whole unit (slot -1; in a longest-first schedule n_dp_x is 0 and every unit is an
// entry). sched holds {start_x, n_dp_x, n_tab_x, first entry} per XCD, then the
// entries. Launches without a table (TABLE false) give XCD x the contiguous units
// [x q + min(x, r), + q + (x < r)) of the n = q 8 + r units, computed in place, in
// order, or with the short last blocks of the segments moved to the end of the share
// (short_last_unit).
template <int D, bool PREFIX, bool TABLE>
__device__ __forceinline__ void fwd_unit(
    int wave, uint32_t x, int pos, const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
    const uint16_t* __restrict__ V, uint16_t* __restrict__ O, const int32_t* __restrict__ items,
    const int32_t* __restrict__ cols, int n_items, int B, int H, int F, int T, int P, int nqb,
    const int32_t* __restrict__ sched, float* __restrict__ ws_o, float* __restrict__ ws_lse,
    float* __restrict__ lse, float* __restrict__ ws_parts, float c, uint32_t qflip, uint32_t qmask,
    uint16_t (&sK)[2][Shape<D>::kTileElems], uint16_t (&sV)[2][Shape<D>::kTileElems]) {
  constexpr int kBlockQ = fwd_rows_per_wg<D>();
  const uint32_t per_b = (uint32_t)n_items * (uint32_t)nqb;
  FwdItem it;
  it.t0 = 0;
  it.nt = -1;
  it.part = -1;
  uint32_t u;
  if constexpr (!TABLE) {
    const uint32_t n = (uint32_t)B * per_b;
    u = share_start(n, x) + (uint32_t)pos;
    // Where every segment ends on a short block that runs on two waves (fwd_tail_rows),
    // the share runs those blocks after its full ones (short_last_unit).
    if constexpr (!PREFIX && (D == 64 || D == 96)) {
      if (nqb > 1 && T - (nqb - 1) * kBlockQ <= 32) u = short_last_unit(n, (uint32_t)nqb, x, (uint32_t)pos);
    }
  } else {
    const int32_t* xi = sched + 4 * x;
    const int n_dp = xi[1];
    if (pos < n_dp) {
      u = (uint32_t)xi[0] + (uint32_t)pos;
    } else {
      const int32_t* pc = sched + 32 + 4 * (xi[3] + pos - n_dp);
      u = (uint32_t)pc[0];
      it.t0 = pc[1];
      it.nt = pc[2];
      it.part = pc[3];
    }
  }
  const Layout<PREFIX> lay{F, T, P};
  it.B = (uint32_t)B;
  it.b = u / per_b;
  const uint32_t rem = u - it.b * per_b;
  const int32_t* item = items + 5 * (rem / nqb);
  it.bh = it.b * (uint32_t)H + (uint32_t)item[0];
  it.frame = item[1];
  it.kbeg = item[2];
  it.n_kept = item[3];
  it.slot = item[4];  // >= 0: a piece of a split frame, written as a partial
  it.qb = (int)(rem % nqb);
  it.cols = cols;
  it.seg0 = lay.start(it.frame);
  it.seg_len = lay.len(it.frame);
  // With a prefix the text segment is shorter than the grid's query blocks assume.
  if (PREFIX && it.qb * kBlockQ >= it.seg_len) return;

  it.head_rows = (size_t)P * PREFIX + (size_t)F * T;
  const size_t head_elems = it.head_rows * D;
  it.Qh = Q + it.bh * head_elems;
  it.Kh = K + it.bh * head_elems;
  it.Vh = V + it.bh * head_elems;
  it.Oh = O + it.bh * head_elems;

  // A query block at the end of a segment with at most 32 valid rows runs on two
  // waves that split the keys of every tile. Not in the d = 96 kernels with a text
  // prefix or a unit table: their epilogues keep more scalars live across the main
  // tile loop, and with this path as well one of them spills to a vector register,
  // which pushes a loader offset of the loop (at 256 VGPRs) into scratch memory. Not
  // at d = 128, whose full blocks already run one column block per wave: there the
  // short blocks gained nothing, and with dense masks they ran ahead of the full
  // blocks of their segment, which then took longer per tile.
  if constexpr (D == 64 || (D == 96 && !PREFIX && !TABLE)) {
    if (it.seg_len - it.qb * kBlockQ <= 32) {
      fwd_tail_rows<D, PREFIX, TABLE>(wave, it, lay, sK, sV, ws_o, ws_lse, lse, ws_parts, c, qflip, qmask);
      return;
    }
  }
  // A query block at the end of a segment with at most 32 valid rows per wave runs
  // with one column block per wave. Only at d = 64: at d = 96 the second instance of
  // the tile loop makes the register allocator spill the main one.
  if constexpr (fwd_q_blocks<D>() == 2 && D == 64) {
    if (it.seg_len - it.qb * kBlockQ <= kWaves * 32) {
      fwd_rows<D, PREFIX, 1, TABLE>(wave, it, lay, sK, sV, ws_o, ws_lse, lse, ws_parts, c, qflip, qmask);
      return;
    }
  }
  fwd_rows<D, PREFIX, fwd_q_blocks<D>(), TABLE>(wave, it, lay, sK, sV, ws_o, ws_lse, lse, ws_parts, c, qflip,
                                                qmask);
}

// The forward kernel's arguments, passed by value (they live in the kernel-argument
// segment, where the work loop reads them again for every unit).
struct FwdKernelArgs {
  const uint16_t* Q;
  const uint16_t* K;
  const uint16_t* V;
  uint16_t* O;
  const int32_t* items;
  const int32_t* cols;
  const int32_t* sched;
  float* ws_o;
  float* ws_lse;
  float* lse;
  float* ws_parts;
  int* queue;
  int n_wg;  // the grid size
  int n_items, B, H, F, T, P, nqb;
  float c;
  uint32_t qflip, qmask;
};

// The kernel. Without PERSIST, one workgroup per queue position: workgroup blockIdx
// takes position blockIdx / 8 of XCD blockIdx % 8 (the hardware hands workgroup ids to
// the eight XCDs in turn), and the in-order dispatcher starts each as a slot frees.
// With PERSIST, a work loop: at most the resident number of workgroups per XCD, each
// taking the next position of its XCD's queue (queue[x], an atomic counter) until the
// queue is exhausted. For the plans the host selects (the MM-DiT form with split
// frames: pieces of the text and global rows, short video units and empty text query
// blocks), the dispatcher leaves slots idle that the loop keeps busy. The queue
// counters start at zero; the last workgroup to finish (counted in queue[8]) sets all
// nine back to zero for the next launch on the same queue. No workgroup ever waits
// for another.
template <int D, bool PREFIX, bool TABLE, bool PERSIST>
__global__ __launch_bounds__(kThreads, 2) void tile_attn_fwd_kernel(const FwdKernelArgs args) {
  using Sh = Shape<D>;
  __shared__ __attribute__((aligned(1024))) uint16_t sK[2][Sh::kTileElems];
  __shared__ __attribute__((aligned(1024))) uint16_t sV[2][Sh::kTileElems];

  const uint32_t x = blockIdx.x % 8;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // Queue positions of XCD y.
  auto positions = [](uint32_t y, int B, int n_items, int nqb, const int32_t* sched) {
    if constexpr (!TABLE) {
      const uint32_t n = (uint32_t)B * (uint32_t)n_items * (uint32_t)nqb;
      return (int)(n / 8 + (y < n % 8 ? 1u : 0u));
    } else {
      return sched[4 * y + 1] + sched[4 * y + 2];
    }
  };
  if constexpr (!PERSIST) {
    const int pos = (int)(blockIdx.x / 8);
    if (pos >= positions(x, args.B, args.n_items, args.nqb, args.sched)) return;
    fwd_unit<D, PREFIX, TABLE>(wave, x, pos, args.Q, args.K, args.V, args.O, args.items, args.cols,
                               args.n_items, args.B, args.H, args.F, args.T, PREFIX ? args.P : 0, args.nqb,
                               args.sched, args.ws_o, args.ws_lse, args.lse, args.ws_parts, args.c, args.qflip,
                               args.qmask, sK, sV);
  } else {
    __shared__ int s_pos[2];
    // The arguments are read from the argument segment where they are needed, through a
    // pointer the compiler cannot see is loop-invariant, so that no argument is held in
    // a scalar register across the loop (the tile loop needs them all); the lane id is
    // read the same way.
    using KArgPtr = const __attribute__((address_space(4))) FwdKernelArgs*;
    auto fresh_args = []() {
      KArgPtr ap = (KArgPtr)__builtin_amdgcn_kernarg_segment_ptr();
      asm volatile("" : "+s"(ap));
      return ap;
    };
    auto first_thread = [&]() {
      int lane;
      asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lane));
      return wave == 0 && lane == 0;
    };
    // s_pos alternates between two words, so thread 0 never overwrites a position
    // another wave has yet to read (one barrier between each write and its reads).
    for (int round = 0;; ++round) {
      KArgPtr ap = fresh_args();
      if (first_thread()) s_pos[round & 1] = atomicAdd(ap->queue + x, 1);
      __syncthreads();
      const int pos = __builtin_amdgcn_readfirstlane(s_pos[round & 1]);
      if (pos >= positions(x, ap->B, ap->n_items, ap->nqb, ap->sched)) break;
      fwd_unit<D, PREFIX, TABLE>(wave, x, pos, ap->Q, ap->K, ap->V, ap->O, ap->items, ap->cols,
                                 ap->n_items, ap->B, ap->H, ap->F, ap->T, PREFIX ? ap->P : 0, ap->nqb,
                                 ap->sched, ap->ws_o, ap->ws_lse, ap->lse, ap->ws_parts, ap->c, ap->qflip,
                                 ap->qmask, sK, sV);
    }
    KArgPtr ap = fresh_args();
    if (first_thread() && atomicAdd(ap->queue + 8, 1) == ap->n_wg - 1) {
#pragma unroll
      for (int i = 0; i < 9; ++i) atomicExch(ap->queue + i, 0);
    }
  }
}

// Combines the parts of query blocks whose kept tiles were shared out among several
// workgroups (the end of each XCD's run); a part's row is D + 4 floats, O/l then its
// log-sum-exp. One thread per (split unit, row of the block, 8 consecutive d): with
// M the largest part log-sum-exp (base 2), O = sum_p
// 2^(lse_p - M) (O/l)_p / sum_p 2^(lse_p - M). A unit of an item that is itself a
// piece of a split frame (item slot >= 0) writes the frame piece's partial row
// (fp32 O/l and base-2 log-sum-exp) for the frame merge; any other writes its output
// row in bf16 (RNE) and the natural-log log-sum-exp.
template <int D>
__global__ __launch_bounds__(256) void merge_parts_kernel(
    const float* __restrict__ ws_parts, const int32_t* __restrict__ cut_units, int n_units,
    const int32_t* __restrict__ items,
    int n_items, int nqb, int rows_per_block, int B, int H, int F, int T, int P,
    uint16_t* __restrict__ O, float* __restrict__ lse, float* __restrict__ ws_o,
    float* __restrict__ ws_lse) {
  constexpr int kGroups = D / 8;
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t per_unit = (size_t)rows_per_block * kGroups;
  if (idx >= per_unit * (size_t)n_units) return;
  const int un = (int)(idx / per_unit);
  const int r = (int)((idx % per_unit) / kGroups), grp = (int)(idx % kGroups);
  const uint32_t u = (uint32_t)cut_units[3 * un];
  const int slot0 = cut_units[3 * un + 1], np = cut_units[3 * un + 2];
  const uint32_t per_b = (uint32_t)n_items * (uint32_t)nqb;
  const uint32_t b = u / per_b, rem = u - b * per_b;
  const int32_t* item = items + 5 * (rem / nqb);
  const int head = item[0], frame = item[1], slot = item[4];
  const int qrow = (int)(rem % nqb) * rows_per_block + r;
  const int seg0 = frame < F ? P + frame * T : 0, seg_len = frame < F ? T : P;
  if (qrow >= seg_len) return;
  float mx = -INFINITY;
  for (int p = 0; p < np; ++p) mx = fmaxf(mx, ws_parts[((size_t)(slot0 + p) * rows_per_block + r) * (D + 4) + D]);
  f32x4 a0 = {0.f, 0.f, 0.f, 0.f}, a1 = {0.f, 0.f, 0.f, 0.f};
  float wsum = 0.f;
  if (mx != -INFINITY) {
    for (int p = 0; p < np; ++p) {
      const float* row = ws_parts + ((size_t)(slot0 + p) * rows_per_block + r) * (D + 4);
      const float w = fast_exp2(row[D] - mx);
      const f32x4* src = reinterpret_cast<const f32x4*>(row + 8 * grp);
      a0 += w * src[0];
      a1 += w * src[1];
      wsum += w;
    }
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  const f32x8 x = {a0[0] * inv, a0[1] * inv, a0[2] * inv, a0[3] * inv,
                   a1[0] * inv, a1[1] * inv, a1[2] * inv, a1[3] * inv};
  const float lse2 = wsum > 0.f ? mx + __builtin_amdgcn_logf(wsum) : -INFINITY;
  if (slot < 0) {
    const size_t orow = (b * H + head) * ((size_t)P + (size_t)F * T) + seg0 + qrow;
    *reinterpret_cast<bf16x8*>(O + orow * D + 8 * grp) = __builtin_convertvector(x, bf16x8);
    if (lse && grp == 0) lse[orow] = lse2 * 0.69314718055994531f;
  } else {
    const size_t prow = ((size_t)slot * B + b) * (size_t)max(T, P) + qrow;
    f32x4* dst = reinterpret_cast<f32x4*>(ws_o + prow * D + 8 * grp);
    dst[0] = f32x4{x[0], x[1], x[2], x[3]};
    dst[1] = f32x4{x[4], x[5], x[6], x[7]};
    if (grp == 0) ws_lse[prow] = lse2;
  }
}

// Combines the pieces of split query frames (or of the split text segment of the
// MM-DiT form). One thread per (split segment, batch entry, row, 8 consecutive d):
// with M the largest piece log-sum-exp, out = sum_p 2^(lse_p - M) (O/l)_p /
// sum_p 2^(lse_p - M), rounded to bf16 (RNE); the row's log-sum-exp is
// M + log2(sum_p 2^(lse_p - M)), stored in natural log. Partials are laid out
// [slot][batch][L][d] with L = max(T, P) rows per slot.
template <int D>
__global__ __launch_bounds__(256) void merge_partials_kernel(
    const float* __restrict__ ws_o, const float* __restrict__ ws_lse,
    const int32_t* __restrict__ heavy, int n_heavy, int B, int H, int F, int T, int P,
    uint16_t* __restrict__ O, float* __restrict__ lse) {
  constexpr int kGroups = D / 8;
  const int L = max(T, P);
  const size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t per_seg = (size_t)B * L * kGroups;
  if (idx >= per_seg * (size_t)n_heavy) return;
  const int hv = (int)(idx / per_seg);
  const size_t r = idx - (size_t)hv * per_seg;
  const int grp = (int)(r % kGroups);
  const size_t row = r / kGroups;  // b * L + t
  const size_t b = row / L, t = row - b * L;
  const int head = heavy[4 * hv], frame = heavy[4 * hv + 1];
  const int slot0 = heavy[4 * hv + 2], np = heavy[4 * hv + 3];
  const int seg0 = frame < F ? P + frame * T : 0, seg_len = frame < F ? T : P;
  if ((int)t >= seg_len) return;
  const size_t slot_stride = (size_t)B * L;
  float mx = -INFINITY;
  for (int p = 0; p < np; ++p) mx = fmaxf(mx, ws_lse[(size_t)(slot0 + p) * slot_stride + row]);
  f32x4 a0 = {0.f, 0.f, 0.f, 0.f}, a1 = {0.f, 0.f, 0.f, 0.f};
  float wsum = 0.f;
  for (int p = 0; p < np; ++p) {
    const size_t pr = (size_t)(slot0 + p) * slot_stride + row;
    const float w = fast_exp2(ws_lse[pr] - mx);
    const f32x4* src = reinterpret_cast<const f32x4*>(ws_o + pr * D + 8 * grp);
    a0 += w * src[0];
    a1 += w * src[1];
    wsum += w;
  }
  const float inv = 1.f / wsum;
  const size_t orow = (b * H + head) * ((size_t)P + (size_t)F * T) + seg0 + t;
  const f32x8 x = {a0[0] * inv, a0[1] * inv, a0[2] * inv, a0[3] * inv,
                   a1[0] * inv, a1[1] * inv, a1[2] * inv, a1[3] * inv};
  *reinterpret_cast<bf16x8*>(O + orow * D + 8 * grp) = __builtin_convertvector(x, bf16x8);
  if (lse && grp == 0) lse[orow] = (mx + __builtin_amdgcn_logf(wsum)) * 0.69314718055994531f;
}

template <int D>
hipError_t launch_d(const FwdArgs& a, hipStream_t stream) {
  const int nqb = (std::max(a.T, a.P) + fwd_rows_per_wg<D>() - 1) / fwd_rows_per_wg<D>();
  // The work loop where the host asks for it (and only at d = 64: at d = 96 it would
  // cost the tile loop registers it does not have); the kernel that can run parts of
  // units only where the schedule has some.
  const bool persist = a.queue != nullptr && a.P > 0 && D == 64;
  const dim3 grid(8u * (uint32_t)(persist ? std::min(a.wg_per_xcd, a.slots_per_xcd) : a.wg_per_xcd));
  auto go = [&](auto prefix, auto table_c) {
    constexpr bool kPrefix = decltype(prefix)::value, kTable = decltype(table_c)::value;
    const FwdKernelArgs ka{a.q,      a.k,   a.v,        a.out,   a.items,         a.cols,
                           a.sched,  a.ws_o, a.ws_lse,  a.lse,   a.ws_parts,      a.queue,
                           (int)grid.x, a.n_items, a.B, a.H,    a.F,             a.T,
                           kPrefix ? a.P : 0, nqb, a.c, a.qflip, a.qmask};
    if (kPrefix && D == 64 && persist)
      hipLaunchKernelGGL((tile_attn_fwd_kernel<D, kPrefix, kTable, kPrefix && D == 64>), grid, dim3(kThreads), 0,
                         stream, ka);
    else
      hipLaunchKernelGGL((tile_attn_fwd_kernel<D, kPrefix, kTable, false>), grid, dim3(kThreads), 0, stream, ka);
  };
  using Y = std::true_type;
  using N = std::false_type;
  const bool table = a.n_cut_units > 0 || a.unit_table;
  if (a.P > 0) {
    if (table) go(Y{}, Y{});
    else go(Y{}, N{});
  } else {
    if (table) go(N{}, Y{});
    else go(N{}, N{});
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_cut_units == 0) return e;
  const size_t threads = (size_t)a.n_cut_units * fwd_rows_per_wg<D>() * (D / 8);
  hipLaunchKernelGGL(merge_parts_kernel<D>, dim3((uint32_t)((threads + 255) / 256)), dim3(256), 0, stream,
                     a.ws_parts, a.cut_units, a.n_cut_units, a.items, a.n_items, nqb,
                     fwd_rows_per_wg<D>(), a.B, a.H, a.F, a.T, a.P, a.out, a.lse, a.ws_o, a.ws_lse);
  return hipGetLastError();
}

template <int D>
hipError_t launch_merge_d(const MergeArgs& a, hipStream_t stream) {
  const size_t threads = (size_t)a.n_heavy * a.B * std::max(a.T, a.P) * (D / 8);
  const size_t blocks = (threads + 255) / 256;
  hipLaunchKernelGGL(merge_partials_kernel<D>, dim3((uint32_t)blocks), dim3(256), 0, stream, a.ws_o,
                     a.ws_lse, a.heavy, a.n_heavy, a.B, a.H, a.F, a.T, a.P, a.out, a.lse);
  return hipGetLastError();
}

}  // namespace

int fwd_rows_per_workgroup(int d) {
  switch (d) {
    case 64: return fwd_rows_per_wg<64>();
    case 96: return fwd_rows_per_wg<96>();
    case 128: return fwd_rows_per_wg<128>();
    default: return 0;
  }
}

hipError_t launch_merge_partials(const MergeArgs& a, hipStream_t stream) {
  switch (a.d) {
    case 64: return launch_merge_d<64>(a, stream);
    case 96: return launch_merge_d<96>(a, stream);
    case 128: return launch_merge_d<128>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_tile_attn_fwd(const FwdArgs& a, hipStream_t stream) {
  switch (a.d) {
    case 64: return launch_d<64>(a, stream);
    case 96: return launch_d<96>(a, stream);
    case 128: return launch_d<128>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace ta
