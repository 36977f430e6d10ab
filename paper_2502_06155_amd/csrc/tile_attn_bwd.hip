// gfx950 (MI355X, CDNA4) kernels for the gradients of tile-sparse 3D attention.
//
// What is computed: the forward pass (Sec. 3.3 of Efficient-vDiT) gives query
// token s the output out_s = sum_t P_st v_t, P_st = softmax over the keys t of the
// frames its frame keeps of scale * <q_s, k_t>. With the upstream gradient dO, the
// forward's row log-sum-exp lse_s and delta_s = <dO_s, out_s>, the chain rule
// through the softmax gives, over kept (s, t) pairs only:
//   P_st = exp(scale <q_s, k_t> - lse_s),  dP_st = <dO_s, v_t>,
//   dS_st = P_st (dP_st - delta_s),
//   dq_s = scale sum_t dS_st k_t,  dk_t = scale sum_s dS_st q_s,  dv_t = sum_s P_st dO_s.
// Stage 3 of the method (Sec. 3.4) trains the sparse model through this; dropped
// tiles are never read here either.
//
// Passes (all on the caller's stream)
//   prep  lse in base 2 and -delta per query row (both gradient kernels start
//         their dP accumulations at -delta, so dP - delta takes no vector op).
//   dq    one workgroup per 128 query rows of a query frame (or of the text with a
//         prefix, see Layout), over the kept key
//         tiles (the forward's work list): S^T = K Q^T, dP^T = V dO^T,
//         dQ^T += K^T dS^T. Each lane owns one query of its wave's 32-query
//         column block, so lse and -delta are per-lane constants.
//   dkdv  one workgroup per 128 key rows of a key frame, over the query tiles of
//         the frames that keep it (the work list of the transposed mask):
//         S = Q K^T, dP = dO V^T, dV^T += dO^T P, dK^T += Q^T dS. Each lane owns
//         one key of its wave's 32-key column block.
//   sum   adds the fp32 partials of frames the work plan split into pieces.
// dq is recomputed in its own pass instead of being accumulated from the key side:
// fp32 atomics from every (key block, query block) pair would move several TB/s
// through L2 at this shape, more than recomputing S and dP costs on the matrix cores.
//
// Both gradient kernels keep one operand of every product in registers (the
// wave's 32 queries or 32 keys) and stream the other through LDS (see kRowsPerWg
// below for why not 64 as in the forward kernel).
//
// LDS layout: every staged tile is read both row-wise (16 bytes per lane, 16
// consecutive rows per access) and transposed (ds_read_b64_tr_b16: 4 consecutive
// rows x 64 bytes per half-wave access), so one XOR swizzle dsw(r) of the 16-byte
// pieces serves both: over 16 consecutive rows it spreads one piece column over
// all 64 banks, and over 4 consecutive rows (starting at a multiple of 4) it puts
// the rows' 64-byte quads in different bank groups.
#include <hip/hip_runtime.h>

#include <type_traits>

#include <float.h>
#include <stdint.h>

#include <algorithm>

#include "launch.h"
#include "tile_common.h"

namespace ta {
namespace {

constexpr int kBwdWaves = 4;
constexpr int kBwdThreads = 64 * kBwdWaves;
// Each wave owns one 32-row column block (32 queries in the dq pass, 32 keys in
// the dk/dv pass). That keeps every operand, accumulator and score in 256 VGPRs,
// so two workgroups share a CU and one wave's softmax-gradient arithmetic overlaps
// the other's matrix instructions. Measured at the 93-frame shape this beats 64
// rows per wave at one workgroup per CU (which halves the LDS fragment reads per
// MFMA but puts the accumulators in AGPRs, copies the scores out of them and
// serialises the vector work) by 17% (dq) and 12% (dk/dv). At d = 128 the dk/dv
// pass needs more than 256 registers and runs one workgroup per CU.
constexpr int kRowsPerWg = kBwdWaves * 32;

// What one launch of the key-side kernel produces. At d = 128 dK and dV together
// (their accumulators, K and V operands alone take 192 registers) need one workgroup
// per CU with the scores copied out of AGPRs; two passes that each fit 256 VGPRs
// (dV: S and P only; dK: S, dP and dS) run at two workgroups per CU and, although
// they form S twice (40 products instead of 32), take less time.
enum KeyPass { kDkDv = 0, kDvOnly = 1, kDkOnly = 2 };
template <int D>
constexpr bool split_key_pass() { return D == 128; }

template <int D>
struct BShape {
  static constexpr int kChunks = D / 16;
  static constexpr int kDBlocks = D / 32;
  static constexpr int kPieces = D / 8;
  static constexpr int kTileElems = kBlockK * D;
  static constexpr int kLoadsPerWave = kBlockK * kPieces / 64 / kBwdWaves;
  static_assert(kBlockK * kPieces == 64 * kBwdWaves * kLoadsPerWave, "whole loads per wave");
};

template <int D>
__device__ __forceinline__ int dsw(int r) {
  if constexpr (D == 64) return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
  else if constexpr (D == 96) return (r >> 2) & 3;
  else return ((r & 3) << 2) | ((r >> 2) & 3);
}
template <int D>
__device__ __forceinline__ int d_slot(int r, int p) { return (r * (D / 8) + (p ^ dsw<D>(r))) * 8; }

// Direct global -> LDS loads of one 64-row tile in the dsw layout (see the
// forward kernel's TileLoader: the XOR only permutes pieces inside a row, and one
// load covers whole rows or aligned quads, so it reads contiguous memory).
template <int D>
struct DualLoader {
  int off[BShape<D>::kLoadsPerWave];
  __device__ __forceinline__ void init(int wave, int lane) {
#pragma unroll
    for (int j = 0; j < BShape<D>::kLoadsPerWave; ++j) {
      const int q = 64 * (wave + kBwdWaves * j) + lane;
      const int r = q / BShape<D>::kPieces, ps = q % BShape<D>::kPieces;
      off[j] = (r * D + 8 * (ps ^ dsw<D>(r))) * 2;
    }
  }
  __device__ __forceinline__ void load(const uint16_t* Xh, size_t row0, int nvalid,
                                       const uint16_t* lds, int wave) const {
    const i32x4 rs = buffer_words(Xh + row0 * D, (uint32_t)(nvalid * D * 2));
    const uint32_t base = lds_addr(lds);
#pragma unroll
    for (int j = 0; j < BShape<D>::kLoadsPerWave; ++j)
      load_to_lds(rs, __builtin_amdgcn_readfirstlane(base + 1024u * (uint32_t)(wave + kBwdWaves * j)),
                  off[j]);
  }
};

// Row-wise fragment offsets (A operand, rows = tile rows): lane (n, h) reads row
// n of a 32-row block, piece 2 cc + h of chunk cc. Row block rb adds rb * 32 * D
// (the swizzle depends only on the low 4 bits of the row).
template <int D>
struct RowAddr {
  // At d = 96 the swizzle only permutes the low two bits of the piece index, so
  // chunks cc and cc + 2 sit 4 pieces apart.
  static constexpr int kN = D == 96 ? 2 : D / 16;
  int at[kN];
  __device__ __forceinline__ void init(int n, int hf) {
#pragma unroll
    for (int cc = 0; cc < kN; ++cc) at[cc] = d_slot<D>(n, 2 * cc + hf);
  }
  __device__ __forceinline__ int get(int cc) const {
    if constexpr (D == 96) return at[cc & 1] + 32 * (cc >> 1);
    else return at[cc];
  }
};

// Transposed fragment offsets (A operand, rows = d, contraction over tile rows):
// lane l (group g = l/16, j = l%16) reads row 4(g/2) + j/4 (lo) and that row + 8
// (hi), d = 32 mb + 16(g%2) + 4(j%4) .. +3. Chunk ch (16 rows) adds 16 ch * D.
template <int D>
struct TrAddr {
  // At d = 96 the swizzle leaves the quad index 4 mb of a piece alone: d-block mb
  // sits 32 mb elements further.
  static constexpr int kN = D == 96 ? 1 : D / 32;
  int lo[kN], hi[kN];
  __device__ __forceinline__ void init(int lane) {
    const int g = lane >> 4, j = lane & 15;
    const int r = 4 * (g >> 1) + (j >> 2);
#pragma unroll
    for (int mb = 0; mb < kN; ++mb) {
      const int p = 4 * mb + 2 * (g & 1) + ((j >> 1) & 1);
      lo[mb] = d_slot<D>(r, p) + 4 * (j & 1);
      hi[mb] = d_slot<D>(r + 8, p) + 4 * (j & 1);
    }
  }
  __device__ __forceinline__ int get_lo(int mb) const { return D == 96 ? lo[0] + 32 * mb : lo[mb]; }
  __device__ __forceinline__ int get_hi(int mb) const { return D == 96 ? hi[0] + 32 * mb : hi[mb]; }
};

template <int D>
__device__ __forceinline__ bf16x8 row_frag(const uint16_t* tile, const RowAddr<D>& ra, int rb, int cc) {
  return as_bf16x8(load16(tile + rb * 32 * D + ra.get(cc)));
}

// 32 d-rows x 16 tile rows: the contraction index k of lane half h maps to tile
// rows 16 ch + 4h + (0..3) and 16 ch + 8 + 4h + (0..3), the order in which a C
// fragment's entries 8c2 .. 8c2+7 hold their rows.
template <int D>
__device__ __forceinline__ bf16x8 tr_frag(const uint16_t* tile, const TrAddr<D>& ta, int mb, int ch) {
  const uint16_t* p = tile + 16 * ch * D;
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + ta.get_lo(mb)));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + ta.get_hi(mb)));
  const u32x2 a = __builtin_bit_cast(u32x2, lo), b = __builtin_bit_cast(u32x2, hi);
  return as_bf16x8(u32x4{a[0], a[1], b[0], b[1]});
}

// B-operand slices of this lane's row (query or key) of a tensor: d = 16 cc + 8h .. +7.
template <int D>
__device__ __forceinline__ void load_row_operand(const uint16_t* row, bool valid, uint32_t keep,
                                                 uint32_t flip, int hf, bf16x8 (&x)[D / 16]) {
#pragma unroll
  for (int cc = 0; cc < D / 16; ++cc) {
    u32x4 w = {0u, 0u, 0u, 0u};
    if (valid) w = (load16(row + 16 * cc + 8 * hf) & keep) ^ flip;
    x[cc] = as_bf16x8(w);
  }
}

// Stores 16 d-values of this lane's row from a transposed accumulator block
// (entry 4i + j holds d = 32 mb + 8i + 4h + j), times s, as bf16 or fp32.
template <int D>
__device__ __forceinline__ void store_row_bf16(uint16_t* row, const f32x16 (&acc)[D / 32], float s, int hf) {
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f32x4 x = {acc[mb][4 * i] * s, acc[mb][4 * i + 1] * s, acc[mb][4 * i + 2] * s,
                       acc[mb][4 * i + 3] * s};
      const bf16x4 y = __builtin_convertvector(x, bf16x4);
      *reinterpret_cast<u32x2*>(row + 32 * mb + 8 * i + 4 * hf) = __builtin_bit_cast(u32x2, y);
    }
}
template <int D>
__device__ __forceinline__ void store_row_f32(float* row, const f32x16 (&acc)[D / 32], float s, int hf) {
#pragma unroll
  for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const f32x4 x = {acc[mb][4 * i] * s, acc[mb][4 * i + 1] * s, acc[mb][4 * i + 2] * s,
                       acc[mb][4 * i + 3] * s};
      *reinterpret_cast<f32x4*>(row + 32 * mb + 8 * i + 4 * hf) = x;
    }
}

// ---------------------------------------------------------------------------
// prep: lse2 = lse * log2(e), ndelta = -<dO, out> (fp32 sum of bf16 products).
// One workgroup per 64 rows: the 256 threads read the rows' 16-byte pieces
// contiguously (coalesced), leave per-piece partial dots in LDS, and 64 threads
// add up one row each.
constexpr int kPrepRows = 64;

template <int D>
__global__ __launch_bounds__(256) void bwd_prep_kernel(const uint16_t* __restrict__ out,
                                                       const uint16_t* __restrict__ dout,
                                                       const float* __restrict__ lse,
                                                       float* __restrict__ lse2,
                                                       float* __restrict__ ndelta, int64_t rows) {
  constexpr int kPieces = D / 8;
  constexpr int kPerThread = kPrepRows * kPieces / 256;
  static_assert(kPrepRows * kPieces == 256 * kPerThread, "whole pieces per thread");
  __shared__ float part[kPrepRows * kPieces];
  const int64_t row0 = (int64_t)blockIdx.x * kPrepRows;
  const int64_t n_rows = rows - row0 < kPrepRows ? rows - row0 : kPrepRows;
  const int64_t base = row0 * D;
#pragma unroll
  for (int j = 0; j < kPerThread; ++j) {
    const int piece = threadIdx.x + 256 * j;  // piece / kPieces = row within the block
    float acc = 0.f;
    if (piece < n_rows * kPieces) {
      const bf16x8 x = as_bf16x8(load16(out + base + 8 * piece));
      const bf16x8 y = as_bf16x8(load16(dout + base + 8 * piece));
#pragma unroll
      for (int e = 0; e < 8; ++e) acc = __builtin_fmaf((float)x[e], (float)y[e], acc);
    }
    part[piece] = acc;
  }
  __syncthreads();
  if (threadIdx.x < n_rows) {
    float acc = 0.f;
#pragma unroll
    for (int c = 0; c < kPieces; ++c) acc += part[threadIdx.x * kPieces + c];
    const int64_t r = row0 + threadIdx.x;
    ndelta[r] = -acc;
    lse2[r] = lse[r] * 1.4426950408889634f;
  }
}

// ---------------------------------------------------------------------------
// P = exp2(c s - lse2) clamped to [0, 1] (the clamp folds into the exponential's
// output modifier). For kept keys the exponent is <= 0 up to rounding, so the clamp
// changes nothing but rounding; it keeps P finite for the rows and keys past a
// tile's valid range, whose zero-filled operands then contribute exactly nothing
// (see the kernels), so no tile needs a mask.
__device__ __forceinline__ float prob(float s, float c, float lse2) {
  return __builtin_amdgcn_fmed3f(fast_exp2(__builtin_fmaf(s, c, -lse2)), 0.f, 1.f);
}

// ---------------------------------------------------------------------------
// dq pass.
//
// dS^T of one 32-key block for one column block, as the B operand of
// dQ^T += K^T dS^T: entries 8c2 .. 8c2+7 of the C fragment. dp already holds
// dP - delta (its accumulation started at -delta).
__device__ __forceinline__ void dq_scores(const f32x16& s, const f32x16& dp, float c, float lse2,
                                          bf16x8 (&ds)[2]) {
#pragma unroll
  for (int c2 = 0; c2 < 2; ++c2) {
    f32x8 x;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float p = prob(s[8 * c2 + e], c, lse2);
      x[e] = p * dp[8 * c2 + e];
    }
    ds[c2] = __builtin_convertvector(x, bf16x8);
  }
}

// The query-side pass over one work unit (b, item, query block).
template <int D, bool PREFIX>
__device__ __forceinline__ void dq_unit(const BwdArgs& a, int nqb, uint32_t work,
                                        uint16_t (&sK)[2][BShape<D>::kTileElems],
                                        uint16_t (&sV)[2][BShape<D>::kTileElems]) {
  using Sh = BShape<D>;
  const uint32_t per_b = (uint32_t)a.n_items_q * (uint32_t)nqb;
  const uint32_t b = work / per_b;
  const uint32_t rem = work - b * per_b;
  const int32_t* item = a.items_q + 5 * (rem / nqb);
  const uint32_t bh = b * (uint32_t)a.H + (uint32_t)item[0];
  const int frame = item[1], kbeg = item[2], n_kept = item[3], slot = item[4];
  const int qb = (int)(rem % nqb);
  const int T = a.T;
  const Layout<PREFIX> lay{a.F, T, a.P};
  const int seg0 = lay.start(frame), seg_len = lay.len(frame);
  // With a prefix the text segment is shorter than the grid's query blocks assume.
  if (PREFIX && qb * kRowsPerWg >= seg_len) return;

  const size_t head_rows = (size_t)a.P * PREFIX + (size_t)a.F * T;
  const uint16_t* Kh = a.k + bh * head_rows * D;
  const uint16_t* Vh = a.v + bh * head_rows * D;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int n = lane & 31, hf = lane >> 5;
  const int qrow = qb * kRowsPerWg + wave * 32 + n;
  const bool wave_active = qb * kRowsPerWg + wave * 32 < seg_len;

  // This lane's query: Q^T and dO^T B-operand slices, its lse (base 2) and -delta,
  // the start of every dP^T accumulation.
  bf16x8 qf[Sh::kChunks], gf[Sh::kChunks];
  const bool valid = qrow < seg_len;
  const size_t qr = (size_t)bh * head_rows + seg0 + qrow;
  load_row_operand<D>(a.q + qr * D, valid, a.keep, a.flip, hf, qf);
  load_row_operand<D>(a.dout + qr * D, valid, ~0u, 0u, hf, gf);
  const float lse2 = valid ? a.lse2[qr] : 0.f;
  const float ndlt = valid ? a.ndelta[qr] : 0.f;
  f32x16 dp_start;
#pragma unroll
  for (int e = 0; e < 16; ++e) dp_start[e] = ndlt;

  f32x16 acc[Sh::kDBlocks];
#pragma unroll
  for (int mb = 0; mb < Sh::kDBlocks; ++mb) acc[mb] = f32x16{};

  const int tpf = (T + kBlockK - 1) / kBlockK;
  int n_tiles = n_kept * tpf;
  if constexpr (PREFIX) {
    // the text segment (index F) sorts last in a kept list
    if (n_kept > 0 && a.cols_q[kbeg + n_kept - 1] == a.F) n_tiles += (a.P + kBlockK - 1) / kBlockK - tpf;
  }
  if (n_tiles > 0) {
    DualLoader<D> ld;
    ld.init(wave, lane);
    RowAddr<D> ra;
    ra.init(n, hf);
    TrAddr<D> ta;
    ta.init(lane);
    SegmentCursor<PREFIX> cur, nxt;
    cur.start(a.cols_q + kbeg, lay);
    ld.load(Kh, cur.key0(), cur.nvalid(), sK[0], wave);
    ld.load(Vh, cur.key0(), cur.nvalid(), sV[0], wave);
    nxt = cur;
    nxt.advance(n_kept);
    wait_tile_loads();
    __syncthreads();

    // S^T and dP^T - delta of 32-key block kb (raw logits; keys past the tile's valid
    // rows read zero rows).
    auto scores = [&](const uint16_t* tk, const uint16_t* tv, int kb, f32x16& sc, f32x16& dp) {
      sc = f32x16{};
      dp = dp_start;
#pragma unroll
      for (int cc = 0; cc < Sh::kChunks; ++cc) {
        sc = mfma32(row_frag<D>(tk, ra, kb, cc), qf[cc], sc);
        dp = mfma32(row_frag<D>(tv, ra, kb, cc), gf[cc], dp);
      }
    };
    // dQ^T += K^T dS^T over block kb.
    auto accumulate = [&](const uint16_t* tk, int kb, const bf16x8 (&ds)[2]) {
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
        for (int mb = 0; mb < Sh::kDBlocks; ++mb)
          acc[mb] = mfma32(tr_frag<D>(tk, ta, mb, 2 * kb + c2), ds[c2], acc[mb]);
    };

    // One tile; the buffer index is a compile-time constant (tiles run in pairs), so
    // every LDS address is a per-lane base plus an immediate offset.
    auto tile_step = [&](auto bufc, int t) {
      constexpr int buf = decltype(bufc)::value;
      if (t + 1 < n_tiles) {
        ld.load(Kh, nxt.key0(), nxt.nvalid(), sK[buf ^ 1], wave);
        ld.load(Vh, nxt.key0(), nxt.nvalid(), sV[buf ^ 1], wave);
      }
      if (wave_active) {
        // Block 1's S/dP run on the matrix cores while block 0's dS forms on the
        // vector ALUs, then block 0's dQ update while block 1's dS forms. The
        // scheduling fences keep each phase's fragments and scores from being
        // hoisted into the previous one (5% faster than leaving the order free).
        f32x16 s0, dp0, s1, dp1;
        bf16x8 ds0[2], ds1[2];
        scores(sK[buf], sV[buf], 0, s0, dp0);
        __builtin_amdgcn_sched_barrier(0);
        scores(sK[buf], sV[buf], 1, s1, dp1);
        dq_scores(s0, dp0, a.c, lse2, ds0);
        __builtin_amdgcn_sched_barrier(0);
        accumulate(sK[buf], 0, ds0);
        dq_scores(s1, dp1, a.c, lse2, ds1);
        __builtin_amdgcn_sched_barrier(0);
        accumulate(sK[buf], 1, ds1);
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

  if (qrow < seg_len) {
    if (slot < 0) {
      store_row_bf16<D>(a.dq + qr * D, acc, a.scale, hf);
    } else {
      const int slot_rows = PREFIX ? max(T, a.P) : T;
      const size_t prow = ((size_t)slot * a.B + b) * slot_rows + qrow;
      store_row_f32<D>(a.ws_dq + prow * D, acc, a.scale, hf);
    }
  }
}

// One workgroup per unit; the ids the hardware sends to one XCD cover a contiguous
// range of units.
template <int D, bool PREFIX>
__global__ __launch_bounds__(kBwdThreads, 2) void bwd_dq_kernel(const BwdArgs a, int nqb) {
  using Sh = BShape<D>;
  __shared__ __attribute__((aligned(1024))) uint16_t sK[2][Sh::kTileElems];
  __shared__ __attribute__((aligned(1024))) uint16_t sV[2][Sh::kTileElems];
  dq_unit<D, PREFIX>(a, nqb, xcd_remap(blockIdx.x, a.n_wg_q), sK, sV);
}

// fn(integral_constant<int, i>) for i = 0 .. N-1, in order.
template <int N, int I = 0, typename Fn>
__device__ __forceinline__ void static_for(Fn&& fn) {
  if constexpr (I < N) {
    fn(std::integral_constant<int, I>{});
    static_for<N, I + 1>(static_cast<Fn&&>(fn));
  }
}

// ---------------------------------------------------------------------------
// dk/dv pass.
// The key-side pass over one work unit (b, item of the transposed plan, key block).
template <int D, bool PREFIX, int MODE>
__device__ __forceinline__ void dkdv_unit(const BwdArgs& a, int nkb, uint32_t work,
                                          uint16_t (&sQ)[2][BShape<D>::kTileElems],
                                          uint16_t (&sG)[2][BShape<D>::kTileElems],
                                          float (&sL)[2][kBlockK], float (&sD)[2][kBlockK]) {
  constexpr bool kWantDv = MODE != kDkOnly, kWantDk = MODE != kDvOnly;
  using Sh = BShape<D>;
  const uint32_t per_b = (uint32_t)a.n_items_k * (uint32_t)nkb;
  const uint32_t b = work / per_b;
  const uint32_t rem = work - b * per_b;
  const int32_t* item = a.items_k + 5 * (rem / nkb);
  const uint32_t bh = b * (uint32_t)a.H + (uint32_t)item[0];
  const int frame = item[1], qbeg = item[2], n_keep = item[3], slot = item[4];
  const int kblk = (int)(rem % nkb);
  const int T = a.T;
  const Layout<PREFIX> lay{a.F, T, a.P};
  const int seg0 = lay.start(frame), seg_len = lay.len(frame);
  if (PREFIX && kblk * kRowsPerWg >= seg_len) return;

  const size_t head_rows = (size_t)a.P * PREFIX + (size_t)a.F * T;
  const uint16_t* Qh = a.q + bh * head_rows * D;
  const uint16_t* Gh = a.dout + bh * head_rows * D;
  const float* Lh = a.lse2 + bh * head_rows;
  const float* Dh = a.ndelta + bh * head_rows;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int n = lane & 31, hf = lane >> 5;
  const int krow = kblk * kRowsPerWg + wave * 32 + n;
  const bool wave_active = kblk * kRowsPerWg + wave * 32 < seg_len;

  // This lane's key as B operand of S = Q K^T and dP = dO V^T.
  bf16x8 kf[Sh::kChunks], vf[kWantDk ? Sh::kChunks : 1];
  const bool valid = krow < seg_len;
  const size_t kr = (size_t)bh * head_rows + seg0 + krow;
  load_row_operand<D>(a.k + kr * D, valid, a.keep, a.flip, hf, kf);
  if constexpr (kWantDk) load_row_operand<D>(a.v + kr * D, valid, ~0u, 0u, hf, vf);

  f32x16 dk[kWantDk ? Sh::kDBlocks : 1], dv[kWantDv ? Sh::kDBlocks : 1];
#pragma unroll
  for (int mb = 0; mb < Sh::kDBlocks; ++mb) {
    if constexpr (kWantDk) dk[mb] = f32x16{};
    if constexpr (kWantDv) dv[mb] = f32x16{};
  }

  const int tpf = (T + kBlockK - 1) / kBlockK;
  int n_tiles = n_keep * tpf;
  if constexpr (PREFIX) {
    if (n_keep > 0 && a.cols_k[qbeg + n_keep - 1] == a.F) n_tiles += (a.P + kBlockK - 1) / kBlockK - tpf;
  }
  if (n_tiles > 0) {
    DualLoader<D> ld;
    ld.init(wave, lane);
    RowAddr<D> ra;
    ra.init(n, hf);
    TrAddr<D> ta;
    ta.init(lane);
    // Q, dO, lse2 and -delta of one 64-query tile; rows past the valid range read
    // as zeros, so they add exactly nothing below (zero Q and dO rows, P <= 1).
    auto load_tile = [&](const SegmentCursor<PREFIX>& tc, int bi) {
      const size_t row0 = tc.key0();
      const int nv = tc.nvalid();
      ld.load(Qh, row0, nv, sQ[bi], wave);
      ld.load(Gh, row0, nv, sG[bi], wave);
      if (wave == 0) {
        load_dword_to_lds(buffer_words(Lh + row0, (uint32_t)(nv * 4)), lds_addr((const uint16_t*)sL[bi]),
                          4 * lane);
        if constexpr (kWantDk)
          load_dword_to_lds(buffer_words(Dh + row0, (uint32_t)(nv * 4)), lds_addr((const uint16_t*)sD[bi]),
                            4 * lane);
      }
    };
    SegmentCursor<PREFIX> cur, nxt;
    cur.start(a.cols_k + qbeg, lay);
    load_tile(cur, 0);
    nxt = cur;
    nxt.advance(n_keep);
    wait_tile_loads();
    __syncthreads();

    // dP - delta of 32-query half qc of the tile: the accumulation starts at the rows' -delta
    // (entry 8 c2 + 4u + j holds query row 32 qc + 16 c2 + 8u + 4h + j), read at the
    // half's first packet.
    auto dp_start = [&](int buf, int qc, f32x16& dp) {
#pragma unroll
      for (int c2 = 0; c2 < 2; ++c2)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const f32x4 d4 = *reinterpret_cast<const f32x4*>(&sD[buf][32 * qc + 16 * c2 + 8 * u + 4 * hf]);
#pragma unroll
          for (int j = 0; j < 4; ++j) dp[8 * c2 + 4 * u + j] = d4[j];
        }
    };
    // One tile; the buffer index is a compile-time constant (the loop below runs tiles
    // in pairs), so every LDS address is a per-lane base plus an immediate offset.
    auto tile_step = [&](auto bufc, int t) {
      constexpr int buf = decltype(bufc)::value;
      if (t + 1 < n_tiles) load_tile(nxt, buf ^ 1);
      if (wave_active) {
        // One stream of MFMAs (8 D/16 per tile for dV and dK together), each in a
        // fenced packet with its share of the vector work; the operand fragment of
        // MFMA i is read from LDS at packet i - 2 into one of three rotating
        // registers (i - 1 and two registers in the dK pass of d = 128), so no MFMA
        // waits on a read issued just before it (3.5% faster than leaving the order to
        // the compiler). Stream: S (and dP) of half 0, S
        // (and dP) of half 1 with half 0's P (and dS) forming, the dV/dK update of
        // half 0 with half 1's P (and dS) forming, the update of half 1. The passes of
        // d = 128 run the same stream: the dV pass (S, P, dV) without dP, dS and dK,
        // the dK pass (S, dP, dS, dK) without P and dV and with each fragment read one
        // packet ahead into two registers (two ahead would need more registers than it
        // has; the stream is 4.5% faster than the compiler's order there).
        constexpr int kC = Sh::kChunks, kMb = Sh::kDBlocks;
        constexpr int kAhead = MODE == kDkOnly ? 1 : 2;  // packets between a read and its use
        constexpr int kHalf = (kWantDk ? 2 : 1) * kC;                   // S (+ dP) MFMAs of a half
        constexpr int kAcc = ((int)kWantDv + (int)kWantDk) * 2 * kMb;  // update MFMAs of a half
        constexpr int kN = 2 * kHalf + 2 * kAcc;                        // the whole stream
        constexpr int kPerC2 = kAcc / 2;                                 // update MFMAs per chunk
        f32x16 sc[2], dp[kWantDk ? 2 : 1];
        bf16x8 pb[kWantDv ? 2 : 1][2], db[kWantDk ? 2 : 1][2];
        f32x4 l4[2][4];  // lse2 of this lane's 16 queries of each half, 4 at a time
        // Update MFMA r of a half: chunk c2, d-block mb, dK (else dV).
        auto upd = [](int r, int& c2, int& mb, bool& is_dk) {
          c2 = r / kPerC2;
          const int q = r % kPerC2;
          if (kWantDv && kWantDk) {
            mb = q / 2;
            is_dk = q % 2;
          } else {
            mb = q;
            is_dk = kWantDk;
          }
        };
        auto frag = [&](auto ic) -> bf16x8 {
          constexpr int i = decltype(ic)::value;
          if constexpr (i < 2 * kHalf) {
            constexpr int h = i / kHalf, r = i % kHalf;
            if constexpr (r < kC) return row_frag<D>(sQ[buf], ra, h, r);
            else return row_frag<D>(sG[buf], ra, h, r - kC);
          } else {
            constexpr int j = i - 2 * kHalf, h = j / kAcc, r = j % kAcc;
            int c2, mb;
            bool is_dk;
            upd(r, c2, mb, is_dk);
            return tr_frag<D>(is_dk ? sQ[buf] : sG[buf], ta, mb, 2 * h + c2);
          }
        };
        auto mfma = [&](auto ic, const bf16x8& f) {
          constexpr int i = decltype(ic)::value;
          if constexpr (i < 2 * kHalf) {
            constexpr int h = i / kHalf, r = i % kHalf;
            if constexpr (r < kC) sc[h] = mfma32(f, kf[r], r == 0 ? f32x16{} : sc[h]);
            else if constexpr (kWantDk) dp[h] = mfma32(f, vf[r - kC], dp[h]);
          } else {
            constexpr int j = i - 2 * kHalf, h = j / kAcc, r = j % kAcc;
            int c2, mb;
            bool is_dk;
            upd(r, c2, mb, is_dk);
            if constexpr (kWantDk && kWantDv) {
              if (is_dk) dk[mb] = mfma32(f, db[h][c2], dk[mb]);
              else dv[mb] = mfma32(f, pb[h][c2], dv[mb]);
            } else if constexpr (kWantDk) {
              dk[mb] = mfma32(f, db[h][c2], dk[mb]);
            } else {
              dv[mb] = mfma32(f, pb[h][c2], dv[mb]);
            }
          }
        };
        // Vector work of packet i: LDS reads of -delta (dP starts) and lse2 ahead of
        // their use, and P (and dS) of half 0 over the second half's S/dP packets, of
        // half 1 over half 0's update packets, 2 queries at a time.
        auto side = [&](auto ic) {
          constexpr int i = decltype(ic)::value;
          if constexpr (kWantDk && (i == 0 || i == kHalf)) dp_start(buf, i / kHalf, dp[i / kHalf]);
          // lse2 of queries 4 q4 .. 4 q4 + 3 (entries 4 q4 ..) of half hh, read two
          // packets before the first packet whose share needs them.
          static_for<8>([&](auto qc) {
            constexpr int hh = decltype(qc)::value / 4, q4 = decltype(qc)::value % 4;
            constexpr int st = hh == 0 ? kHalf : 2 * kHalf, pk = hh == 0 ? kHalf : kAcc;
            constexpr int at = st + ((2 * q4 + 1) * pk + 7) / 8 - 1 - kAhead;
            if constexpr (at == i)
              l4[hh][q4] = *reinterpret_cast<const f32x4*>(&sL[buf][32 * hh + 16 * (q4 / 2) + 8 * (q4 % 2) + 4 * hf]);
          });
          constexpr int h = i < kHalf ? -1 : (i < 2 * kHalf ? 0 : (i < 2 * kHalf + kAcc ? 1 : -1));
          if constexpr (h >= 0) {
            constexpr int k = h == 0 ? i - kHalf : i - 2 * kHalf;  // packet within the share
            constexpr int kPk = h == 0 ? kHalf : kAcc;
#pragma unroll
            for (int u = k * 8 / kPk; u < (k + 1) * 8 / kPk; ++u) {
              // queries e, e+1 of the half: entry e = 8 c2 + 4 uu + j
              const int e = 2 * u, c2 = e / 8, uu = (e % 8) / 4, j = e % 4;
              const float p0 = prob(sc[h][e], a.c, l4[h][2 * c2 + uu][j]);
              const float p1 = prob(sc[h][e + 1], a.c, l4[h][2 * c2 + uu][j + 1]);
              if constexpr (kWantDv) {
                const f32x2 pp = {p0, p1};
                const bf16x2 pq = __builtin_convertvector(pp, bf16x2);
                u32x4 pw = __builtin_bit_cast(u32x4, pb[h][c2]);
                pw[(e % 8) / 2] = __builtin_bit_cast(uint32_t, pq);
                pb[h][c2] = __builtin_bit_cast(bf16x8, pw);
              }
              if constexpr (kWantDk) {
                const f32x2 dd = {p0 * dp[h][e], p1 * dp[h][e + 1]};
                const bf16x2 dq = __builtin_convertvector(dd, bf16x2);
                u32x4 dw = __builtin_bit_cast(u32x4, db[h][c2]);
                dw[(e % 8) / 2] = __builtin_bit_cast(uint32_t, dq);
                db[h][c2] = __builtin_bit_cast(bf16x8, dw);
              }
            }
          }
        };
        bf16x8 fr[kAhead + 1];
        static_for<kAhead>([&](auto jc) {
          constexpr int j = decltype(jc)::value;
          fr[j] = frag(std::integral_constant<int, j>{});
        });
        __builtin_amdgcn_sched_barrier(0);
        static_for<kN>([&](auto ic) {
          constexpr int i = decltype(ic)::value;
          if constexpr (i + kAhead < kN)
            fr[(i + kAhead) % (kAhead + 1)] = frag(std::integral_constant<int, i + kAhead>{});
          mfma(ic, fr[i % (kAhead + 1)]);
          side(ic);
          __builtin_amdgcn_sched_barrier(0);
        });
      }
      cur = nxt;
      nxt.advance(n_keep);
      wait_tile_loads();
      __syncthreads();
    };
    for (int t = 0; t < n_tiles; t += 2) {
      tile_step(std::integral_constant<int, 0>{}, t);
      if (t + 1 < n_tiles) tile_step(std::integral_constant<int, 1>{}, t + 1);
    }
  }

  // dK uses the unflipped q of the LDS tiles, so scale (with its sign) applies.
  if (krow < seg_len) {
    if (slot < 0) {
      if constexpr (kWantDk) store_row_bf16<D>(a.dk + kr * D, dk, a.scale, hf);
      if constexpr (kWantDv) store_row_bf16<D>(a.dv + kr * D, dv, 1.f, hf);
    } else {
      const int slot_rows = PREFIX ? max(T, a.P) : T;
      const size_t prow = ((size_t)slot * a.B + b) * slot_rows + krow;
      if constexpr (kWantDk) store_row_f32<D>(a.ws_dk + prow * D, dk, a.scale, hf);
      if constexpr (kWantDv) store_row_f32<D>(a.ws_dv + prow * D, dv, 1.f, hf);
    }
  }
}

// One workgroup per unit, as in the query-side pass. (The unit body is a separate
// function in both passes; compiled so, the d = 128 dK pass fits 256 VGPRs without the
// two spilled registers it had as one kernel body, 1.2% faster.)
template <int D, bool PREFIX, int MODE>
__global__ __launch_bounds__(kBwdThreads, 2) void bwd_dkdv_kernel(const BwdArgs a, int nkb) {
  using Sh = BShape<D>;
  __shared__ __attribute__((aligned(1024))) uint16_t sQ[2][Sh::kTileElems];
  __shared__ __attribute__((aligned(1024))) uint16_t sG[2][Sh::kTileElems];
  __shared__ __attribute__((aligned(256))) float sL[2][kBlockK];
  __shared__ __attribute__((aligned(256))) float sD[2][kBlockK];
  dkdv_unit<D, PREFIX, MODE>(a, nkb, xcd_remap(blockIdx.x, a.n_wg_k), sQ, sG, sL, sD);
}

// ---------------------------------------------------------------------------
// Sum of the partials of split segments: one thread per (split segment, batch
// entry, row, 8 consecutive d), rounded to bf16 (RNE). Partials are laid out
// [slot][batch][L][d] with L = max(T, P) rows per slot (T without a prefix).
template <int D>
__global__ __launch_bounds__(256) void sum_partials_kernel(const float* __restrict__ ws,
                                                           const int32_t* __restrict__ heavy,
                                                           int n_heavy, int B, int H, int F, int T,
                                                           int P, uint16_t* __restrict__ out) {
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
  f32x4 a0 = {0.f, 0.f, 0.f, 0.f}, a1 = {0.f, 0.f, 0.f, 0.f};
  for (int p = 0; p < np; ++p) {
    const f32x4* src =
        reinterpret_cast<const f32x4*>(ws + ((size_t)(slot0 + p) * slot_stride + row) * D + 8 * grp);
    a0 += src[0];
    a1 += src[1];
  }
  const size_t orow = (b * H + head) * ((size_t)P + (size_t)F * T) + seg0 + t;
  const f32x8 x = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
  *reinterpret_cast<bf16x8*>(out + orow * D + 8 * grp) = __builtin_convertvector(x, bf16x8);
}

template <int D>
hipError_t prep_d(const PrepArgs& a, hipStream_t stream) {
  const int64_t blocks = (a.rows + kPrepRows - 1) / kPrepRows;
  hipLaunchKernelGGL(bwd_prep_kernel<D>, dim3((uint32_t)blocks), dim3(256), 0, stream, a.out, a.dout,
                     a.lse, a.lse2, a.ndelta, a.rows);
  return hipGetLastError();
}

template <int D>
hipError_t dq_d(const BwdArgs& a, hipStream_t stream) {
  const int nqb = (std::max(a.T, a.P) + kRowsPerWg - 1) / kRowsPerWg;
  if (a.P > 0)
    hipLaunchKernelGGL((bwd_dq_kernel<D, true>), dim3(a.n_wg_q), dim3(kBwdThreads), 0, stream, a, nqb);
  else
    hipLaunchKernelGGL((bwd_dq_kernel<D, false>), dim3(a.n_wg_q), dim3(kBwdThreads), 0, stream, a, nqb);
  return hipGetLastError();
}

template <int D, bool PREFIX, int MODE>
void dkdv_launch(const BwdArgs& a, int nkb, hipStream_t stream) {
  hipLaunchKernelGGL((bwd_dkdv_kernel<D, PREFIX, MODE>), dim3(a.n_wg_k), dim3(kBwdThreads), 0, stream,
                     a, nkb);
}

template <int D, bool PREFIX>
void dkdv_passes(const BwdArgs& a, int nkb, hipStream_t stream) {
  if constexpr (split_key_pass<D>()) {
    dkdv_launch<D, PREFIX, kDvOnly>(a, nkb, stream);
    dkdv_launch<D, PREFIX, kDkOnly>(a, nkb, stream);
  } else {
    dkdv_launch<D, PREFIX, kDkDv>(a, nkb, stream);
  }
}

template <int D>
hipError_t dkdv_d(const BwdArgs& a, hipStream_t stream) {
  const int nkb = (std::max(a.T, a.P) + kRowsPerWg - 1) / kRowsPerWg;
  if (a.P > 0) dkdv_passes<D, true>(a, nkb, stream);
  else dkdv_passes<D, false>(a, nkb, stream);
  return hipGetLastError();
}

template <int D>
hipError_t sum_d(const SumArgs& a, hipStream_t stream) {
  const size_t threads = (size_t)a.n_heavy * a.B * std::max(a.T, a.P) * (D / 8);
  const size_t blocks = (threads + 255) / 256;
  hipLaunchKernelGGL(sum_partials_kernel<D>, dim3((uint32_t)blocks), dim3(256), 0, stream, a.ws,
                     a.heavy, a.n_heavy, a.B, a.H, a.F, a.T, a.P, a.out);
  return hipGetLastError();
}

}  // namespace

int bwd_queries_per_workgroup(int) { return kRowsPerWg; }

int bwd_keys_per_workgroup(int) { return kRowsPerWg; }

#define TA_DISPATCH_D(fn, a, stream)          \
  switch ((a).d) {                            \
    case 64: return fn<64>(a, stream);        \
    case 96: return fn<96>(a, stream);        \
    case 128: return fn<128>(a, stream);      \
    default: return hipErrorInvalidValue;     \
  }

hipError_t launch_bwd_prep(const PrepArgs& a, hipStream_t stream) { TA_DISPATCH_D(prep_d, a, stream) }
hipError_t launch_bwd_dq(const BwdArgs& a, hipStream_t stream) { TA_DISPATCH_D(dq_d, a, stream) }
hipError_t launch_bwd_dkdv(const BwdArgs& a, hipStream_t stream) { TA_DISPATCH_D(dkdv_d, a, stream) }
hipError_t launch_sum_partials(const SumArgs& a, hipStream_t stream) { TA_DISPATCH_D(sum_d, a, stream) }

#undef TA_DISPATCH_D

}  // namespace ta
