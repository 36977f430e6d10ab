// Device helpers shared by the gfx950 tile-attention kernels: vector types, the
// bf16 matrix instruction, wave-uniform tile walking, lane-pair reductions and the
// direct global -> LDS buffer loads.
#pragma once
#include <hip/hip_runtime.h>

#include <stdint.h>

namespace ta {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kBlockK = 64;  // tokens per K/V (or Q/dO) tile staged in LDS

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

// Token layout of one (batch, head). Without a prefix: F frames of T tokens,
// segment j = frame j at j*T. With a prefix (the MM-DiT form): P text tokens first,
// then the frames, so segment j < F starts at P + j*T and segment F is the text,
// P tokens at 0.
template <bool PREFIX>
struct Layout {
  int F, T, P;
  // Written as arithmetic on the fields' values: a conditional choice between two
  // fields can become a load through a chosen address, which keeps the whole
  // struct (and a cursor holding it) in scratch memory instead of registers.
  __device__ __forceinline__ int start(int j) const {
    if constexpr (PREFIX) return (j < F) * (P + j * T);
    else return j * T;
  }
  __device__ __forceinline__ int len(int j) const {
    if constexpr (PREFIX) return P + (j < F) * (T - P);
    else return T;
  }
};

// Walks the 64-token tiles of a list of segments (frames, and the text segment with
// a prefix) in order: tile (e, kt) covers tokens [64 kt, 64 kt + 64) of segment
// cols[e]. All state is wave-uniform (SGPRs); the list is read with one scalar load
// per segment.
template <bool PREFIX>
struct SegmentCursor {
  const int32_t* cols;
  Layout<PREFIX> L;
  int e = 0, kt = 0, kf = 0, tiles = 0;
  __device__ __forceinline__ void start(const int32_t* c, Layout<PREFIX> lay) {
    cols = c;
    L = lay;
    e = 0;
    kt = 0;
    kf = cols[0];
    tiles = (L.len(kf) + kBlockK - 1) / kBlockK;
  }
  __device__ __forceinline__ void advance(int n_segments) {
    if (++kt == tiles) {
      kt = 0;
      if (++e < n_segments) {
        kf = cols[e];
        tiles = (L.len(kf) + kBlockK - 1) / kBlockK;
      }
    }
  }
  // Moves on by n tiles (n >= 0 and within the list).
  __device__ __forceinline__ void skip(int n, int n_segments) {
    while (n >= tiles - kt && e + 1 < n_segments) {
      n -= tiles - kt;
      kt = 0;
      kf = cols[++e];
      tiles = (L.len(kf) + kBlockK - 1) / kBlockK;
    }
    kt += n;
  }
  __device__ __forceinline__ size_t key0() const { return (size_t)L.start(kf) + kt * kBlockK; }
  __device__ __forceinline__ int nvalid() const { return min(kBlockK, L.len(kf) - kt * kBlockK); }
};

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

// Buffer resource words (raw buffer, no stride) over `bytes` bytes at `base`;
// loads past the end return zero, which keeps tile loads inside their frame. The
// base and size are wave-uniform (one tile per workgroup); readfirstlane states so,
// which keeps the descriptor in SGPRs even where the compiler cannot prove it.
__device__ __forceinline__ i32x4 buffer_words(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return i32x4{__builtin_amdgcn_readfirstlane((int)(uint32_t)a),
               __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xffffu)),
               __builtin_amdgcn_readfirstlane((int)bytes), 0x00020000};
}

// One 16-byte-per-lane buffer load written straight to LDS: lane L's 16 bytes
// from byte offset voff land at LDS byte address lds + 16 L. Issued as inline
// assembly so that the compiler does not order every later LDS read behind it;
// completion is awaited explicitly with wait_tile_loads() before the barrier
// that publishes the tile.
__device__ __forceinline__ void load_to_lds(i32x4 rsrc, uint32_t lds, int voff) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %1, %2, 0 offen lds"
      :
      : "s"(lds), "v"(voff), "s"(rsrc)
      : "memory", "m0");
}

// The same with 4 bytes per lane: lane L's dword lands at LDS byte address lds + 4 L.
__device__ __forceinline__ void load_dword_to_lds(i32x4 rsrc, uint32_t lds, int voff) {
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "buffer_load_dword %1, %2, 0 offen lds"
      :
      : "s"(lds), "v"(voff), "s"(rsrc)
      : "memory", "m0");
}

// Waits until every buffer load of this wave, including those writing LDS, is done.
__device__ __forceinline__ void wait_tile_loads() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ uint32_t lds_addr(const uint16_t* p) {
  return __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) uint16_t*)p));
}

// Scheduling hint for a region holding N_MFMA matrix instructions and about
// N_MFMA * VALU_PER vector instructions that do not depend on them: each MFMA is
// followed by VALU_PER vector instructions, so the vector ALUs issue while the
// matrix core runs (LDS reads are left to the scheduler). Used between scheduling
// fences that keep the region to those instructions.
template <int N_MFMA, int VALU_PER>
__device__ __forceinline__ void spread_valu_over_mfma() {
#pragma unroll
  for (int i = 0; i < N_MFMA; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);         // MFMA
    __builtin_amdgcn_sched_group_barrier(0x002, VALU_PER, 0);  // VALU
  }
}

}  // namespace
}  // namespace ta
