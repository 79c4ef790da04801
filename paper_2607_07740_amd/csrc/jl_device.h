// jl_device.h -- device-side building blocks shared by the gfx950 kernels:
// the integer schedule of Jet-Long (arXiv 2607.07740, Sec. 3.1 Eqs. (2)-(3),
// Sec. 3.2 Eq. (5)), the tile classification of Eq. (1)'s window boundary, and
// small wave-level helpers (bf16 packing, lane exchange, transposing LDS read).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace jl {

constexpr int kHeadDim = 128;
constexpr int kHalf = 64;  // rotate-half partner offset and number of RoPE frequencies

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- schedule
// Eq. (2): G = max(1, ceil(L / w)).  Integer ceiling, no floating point.
__host__ __device__ inline int group_size(int L, int w) {
  if (L <= w) return 1;
  return (int)(((int64_t)L + w - 1) / w);
}
// Division by the run-time constant G without a divide instruction
// (Granlund-Montgomery, round-up multiplier with the add-and-shift fix-up):
// with l = ceil(log2 d) and m = floor(2^32 (2^l - d) / d) + 1,
//   t = mulhi(m, x),  x / d = (t + ((x - t) >> 1)) >> (l - 1)
// exactly, for every 32-bit unsigned x and d >= 2 (d = 1 is the identity).
struct FastDiv {
  uint32_t m, l, d;
};

__host__ __device__ inline FastDiv make_fastdiv(uint32_t d) {
  FastDiv f;
  f.d = d;
  f.m = 0;
  f.l = 0;
  if (d <= 1) return f;
  uint32_t l = 0;
  while ((1u << l) < d) ++l;
  f.m = (uint32_t)(((((uint64_t)1 << l) - d) << 32) / d + 1);
  f.l = l;
  return f;
}

__host__ __device__ inline uint32_t fastdiv(uint32_t x, FastDiv f) {
  if (f.d <= 1) return x;
  const uint32_t t = (uint32_t)(((uint64_t)f.m * x) >> 32);
  return (t + ((x - t) >> 1)) >> (f.l - 1);
}

// The same quotient for d >= 2 only, without the d = 1 branch (straight-line
// code for kernels that are launched with G >= 2).  For d = 1 the value is
// meaningless but defined (the shift count is taken mod 32, as the hardware
// shift does), so callers may form it and discard it.
__host__ __device__ inline uint32_t fastdiv_ge2(uint32_t x, FastDiv f) {
  const uint32_t t = (uint32_t)(((uint64_t)f.m * x) >> 32);
  return (t + ((x - t) >> 1)) >> ((f.l - 1) & 31);
}

// Eq. (3): f(x) = floor(x / G) for x >= 0 (truncating division is the floor).
__host__ __device__ inline int remote_pos(int x, FastDiv G) { return (int)fastdiv((uint32_t)x, G); }
// Eq. (5): Delta(x) = f(x) - x.
__host__ __device__ inline int pos_offset(int x, FastDiv G) { return remote_pos(x, G) - x; }

// Key tiles a query block [q0, q1] visits (Eq. (1): a causal pair is local
// iff q - k <= w0, remote iff q - k > w0).  Tiles are BK keys wide.
//   n_kt  tiles up to the block's last query (all others hold no causal pair)
//   n_r   tiles [0, n_r) hold at least one remote pair: k0 < q1 - w0
//   kt_l  tiles [kt_l, n_kt) hold at least one band pair: k0 + BK - 1 >= q0 - w0
struct VisitRanges {
  int n_kt, n_r, kt_l;
};

__host__ __device__ inline VisitRanges visit_ranges(int q0, int q1, int w0, int BK) {
  VisitRanges r;
  r.n_kt = q1 / BK + 1;
  r.n_r = q1 - w0 > 0 ? (q1 - w0 + BK - 1) / BK : 0;
  r.kt_l = q0 - w0 > 0 ? (q0 - w0) / BK : 0;
  return r;
}

// Tile classes: the set of element classes among a tile's causal pairs.
enum TileClass : int { kSkip = 0, kLocal = 1, kRemote = 2, kMixed = 3 };

__host__ __device__ inline int tile_class(const VisitRanges& r, int kt) {
  if (kt >= r.n_kt) return kSkip;
  return (kt >= r.kt_l ? kLocal : 0) | (kt < r.n_r ? kRemote : 0);
}

// ------------------------------------------------------------ wave helpers
__device__ inline float bf16_lo(unsigned w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(unsigned w) { return __uint_as_float(w & 0xffff0000u); }

// Unpack 8 bf16 (one 16-byte vector) to fp32.
__device__ inline void unpack8(const u32x4 v, float* f) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    f[2 * j] = bf16_lo(v[j]);
    f[2 * j + 1] = bf16_hi(v[j]);
  }
}

// Pack 8 fp32 to bf16 with round-to-nearest-even (hardware conversion).
__device__ inline bf16x8 pack8(const float* f) {
  f32x8 t;
#pragma unroll
  for (int j = 0; j < 8; ++j) t[j] = f[j];
  return __builtin_convertvector(t, bf16x8);
}

// Exchange a 16-byte vector with the lane 8 positions away inside its 16-lane
// row (lane i <-> lane i ^ 8), via DPP row rotation.
__device__ inline u32x4 swap_half_row(u32x4 v) {
  u32x4 r;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    r[j] = (unsigned)__builtin_amdgcn_update_dpp((int)0, (int)v[j], 0x128 /* row_ror:8 */, 0xf,
                                                 0xf, false);
  return r;
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Transposing LDS read (gfx950 ds_read_b64_tr_b16).  Inside each 16-lane group
// lane j supplies the address of 4 consecutive 16-bit elements; lane i receives
// element i of each of the 4 lane quads.  With lane j pointing at
// M[r0 + j/4][c0 + 4*(j%4)], lane i receives M[r0 + s][c0 + i] for s = 0..3:
// one column of a 4 x 16 block of a row-major matrix.
__device__ inline i16x4 lds_read_tr4(const void* lds_ptr) {
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_i16x4*)(__attribute__((address_space(3))) void*)(lds_ptr));
}

__device__ inline bf16x8 concat_tr(i16x4 a, i16x4 b) {
  typedef short i16x8 __attribute__((ext_vector_type(8)));
  i16x8 r = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return __builtin_bit_cast(bf16x8, r);
}

__device__ inline f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ inline f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ inline u32x4 load16(const void* p) { return *(const u32x4*)p; }

// Two rotate-half pairs by v_dot2_f32_bf16 (exact bf16 products, one fp32
// rounding each), rounded to bf16 and packed.  From the raw words
// wl = (x_a, x_b), wh = (x_{a+64}, x_{b+64}) and the bf16 (cos, sin) of
// frequencies a and b (cs_a, cs_b):
//   lo = (x_a cos_a - x_{a+64} sin_a,  x_b cos_b - x_{b+64} sin_b)
//   hi = (x_{a+64} cos_a + x_a sin_a,  x_{b+64} cos_b + x_b sin_b)
// The block keeps its own wait states between the permutes and the dot
// instructions and between the dots and the conversions that read them (the
// compiler's hazard tracking does not look inside assembly); its results come
// from ordinary VALU conversions.
__device__ inline void rot_word_dot2(uint32_t wl, uint32_t wh, uint32_t cs_a, uint32_t cs_b,
                                     uint32_t& lo, uint32_t& hi) {
  float a0, a1, b0, b1;
  uint32_t p0, q0, p1, q1;
  asm("v_perm_b32 %6, %11, %10, %14\n\t"   // (x_a, x_a+64)
      "v_perm_b32 %7, %11, %10, %15\n\t"   // (x_a+64, x_a)
      "v_perm_b32 %8, %11, %10, %16\n\t"   // (x_b, x_b+64)
      "v_perm_b32 %9, %11, %10, %17\n\t"   // (x_b+64, x_b)
      "s_nop 1\n\t"
      "v_dot2_f32_bf16 %2, %6, %12, 0 neg_hi:[0,1,0]\n\t"
      "v_dot2_f32_bf16 %3, %8, %13, 0 neg_hi:[0,1,0]\n\t"
      "v_dot2_f32_bf16 %4, %7, %12, 0\n\t"
      "v_dot2_f32_bf16 %5, %9, %13, 0\n\t"
      "s_nop 2\n\t"
      "v_cvt_pk_bf16_f32 %0, %2, %3\n\t"
      "v_cvt_pk_bf16_f32 %1, %4, %5"
      : "=&v"(lo), "=&v"(hi), "=&v"(a0), "=&v"(a1), "=&v"(b0), "=&v"(b1), "=&v"(p0), "=&v"(q0),
        "=&v"(p1), "=&v"(q1)
      : "v"(wl), "v"(wh), "v"(cs_a), "v"(cs_b), "s"(0x05040100u), "s"(0x01000504u),
        "s"(0x07060302u), "s"(0x03020706u));
}

// ------------------------------------------------- direct-to-LDS staging
// Byte address of a __shared__ object inside the workgroup's LDS window.
__device__ inline uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}

// Asynchronous copy of 16 bytes per lane from global memory straight into LDS
// (global_load_lds_dwordx4): lane i's 16 bytes land at lds_base + 16 i, so one
// call moves 1 KB per wave and each lane picks its own source address.
// lds_base must be wave-uniform.  Completion is tracked by the vector-memory
// counter alone: call wait_vmem() before the bytes are read.  Inline assembly
// keeps the compiler from adding a conservative wait in front of every LDS
// read that follows the copy.
// The compiler loads M0 itself (operand constraint); the s_nop is the wait
// state an LDS-bound load needs after an M0 write.
// The base is wave-uniform and 64-bit, in scalar registers, with a 32-bit
// per-lane byte offset; imm is added to both the global and the LDS address.
template <int imm = 0>
__device__ inline void dma16_s(const void* sbase, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 offset:%2"
               :
               : "v"(voff), "s"(sbase), "i"(imm), "{m0}"(lds_base)
               : "memory");
}
// The same copy with the nontemporal hint, for data that is read exactly once.
template <int imm = 0>
__device__ inline void dma16_s_nt(const void* sbase, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 offset:%2 nt"
               :
               : "v"(voff), "s"(sbase), "i"(imm), "{m0}"(lds_base)
               : "memory");
}
__device__ inline void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// Wait until at most N of this wave's vector-memory operations are in flight
// (they complete in issue order, so everything older than the last N is done).
template <int N>
__device__ inline void wait_vmem_n() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"i"(N) : "memory");
}

}  // namespace jl
