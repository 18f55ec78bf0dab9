// Device helpers for the gfx950 kernels: vector types, bf16 packing, MFMA
// wrappers and wavefront exchanges.
//
// MFMA operand layout used throughout (v_mfma_f32_32x32x16_bf16, wave64):
//   A (32 x 16, M x K): lane l holds row l%32, k = 8*(l/32) .. +7
//   B (16 x 32, K x N): lane l holds column l%32, k = 8*(l/32) .. +7
//   C (32 x 32):        lane l holds column l%32, rows
//                       8*(v/4) + 4*(l/32) + (v%4) for v = 0..15
// The reduction index k is free to be permuted as long as A and B agree; the
// kernels exploit that to feed an accumulator straight back as an operand.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

namespace ba {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// The same MFMA with its accumulator pinned to the accumulation registers
// (AGPRs), for long-lived accumulators that only MFMAs touch: the compiler
// then keeps them there instead of moving them between register files.  It
// does not see this as an MFMA, so the caller guarantees the hazards it
// would otherwise pad: the A/B operands are not written by a VALU
// instruction within two wait states (kPad pads them with s_nop 1; callers
// whose schedule keeps the producing instruction slots away pass false, and
// the generated code is checked for it), no other MFMA writes the
// accumulator within the latency of this one, and mfma_drain() separates
// the last one from any VALU read or move of the accumulator.
template <bool kPad = true>
__device__ __forceinline__ void mfma32_acc(f32x16& acc, const bf16x8& a, const bf16x8& b) {
  if constexpr (kPad)
    asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
  else
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// MFMA with a vector-register accumulator and the B operand held in the
// accumulation registers (so long-lived B operands do not occupy vector
// registers).  Opaque to the hazard recognizer: the caller keeps the result
// away from vector-ALU reads until the MFMA has completed (mfma_drain, or
// enough later instructions) and does not write the A operand just before.
__device__ __forceinline__ void mfma32_v_first(f32x16& d, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(d) : "v"(a), "a"(b));
}
__device__ __forceinline__ void mfma32_v(f32x16& d, const bf16x8& a, const bf16x8& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(d) : "v"(a), "a"(b));
}
// mfma32_v_first with the accumulation starting from c (vector registers);
// s_nop 1 pads an addend just written by a vector instruction (kPad false:
// the addend was written long before, e.g. a loop-invariant value).
template <bool kPad = true>
__device__ __forceinline__ void mfma32_v_init(f32x16& d, const bf16x8& a, const bf16x8& b, const f32x16& c) {
  if constexpr (kPad)
    asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %3" : "=&v"(d) : "v"(a), "a"(b), "v"(c));
  else
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %3" : "=&v"(d) : "v"(a), "a"(b), "v"(c));
}

// 16-byte global load straight into accumulation registers (for MFMA
// operands that stay resident there).  Untracked by the compiler: the caller
// waits on the vector-memory counter before the first use.
__device__ __forceinline__ void load16_agpr(bf16x8& d, const bf16* src) {
  asm volatile("global_load_dwordx4 %0, %1, off" : "=a"(d) : "v"(src) : "memory");
}

// A zero accumulator produced in the accumulation registers (an MFMA of zero
// operands with a zero addend), so a loop-carried accumulator never has a
// definition outside them.
__device__ __forceinline__ void mfma32_acc_zero(f32x16& acc) {
  const bf16x8 z = bf16x8{};
  asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %1, 0" : "=a"(acc) : "v"(z));
}
// Rescale an accumulator held in the accumulation registers by a per-lane
// factor.  Empty asm statements with accumulation-register operands bracket
// the vector-ALU multiply, so the accumulator keeps a single register class
// and the compiler neither hoists the reads nor copies it elsewhere.  Call
// between two mfma_drain().
__device__ __forceinline__ void acc_scale(f32x16& acc, float alpha) {
  asm volatile("" : "+a"(acc));  // the reads below stay here, not hoisted
  const f32x16 t = acc * alpha;
  asm volatile("" : "=a"(acc) : "0"(t));
}
// Marks an accumulation-register value as redefined here: vector-ALU uses
// after this point cannot be moved (or copied out) before it.  Place after
// mfma_drain().
__device__ __forceinline__ void acc_settle(f32x16& acc) { asm volatile("" : "+a"(acc)); }
// The same for a vector-register MFMA result of mfma32_v: reads after it
// cannot be hoisted above a preceding mfma_drain().
__device__ __forceinline__ void vacc_settle(f32x16& acc) { asm volatile("" : "+v"(acc)); }
__device__ __forceinline__ void mfma_drain() { asm volatile("s_nop 15\n\ts_nop 15\n\ts_nop 15" ::: "memory"); }

__device__ __forceinline__ bf16x8 ld16(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }
__device__ __forceinline__ void st16(bf16* p, const bf16x8& v) { *reinterpret_cast<bf16x8*>(p) = v; }

__device__ __forceinline__ bf16x8 pack8(float a0, float a1, float a2, float a3, float a4, float a5,
                                         float a6, float a7) {
  bf16x8 r;
  r[0] = (bf16)a0; r[1] = (bf16)a1; r[2] = (bf16)a2; r[3] = (bf16)a3;
  r[4] = (bf16)a4; r[5] = (bf16)a5; r[6] = (bf16)a6; r[7] = (bf16)a7;
  return r;
}

// Two floats rounded to bf16 (nearest even) in one 32-bit word, lo in the
// low half: one v_cvt_pk_bf16_f32 (two scalar casts combined afterwards can
// compile to a conversion each plus a byte permute).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 b16x2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, b16x2));
}

// c + <a, b> over eight bf16 pairs with fp32 products and sums, as four
// packed two-term dot products (v_dot2c_f32_bf16) instead of sixteen
// conversions and eight fused multiply-adds
__device__ __forceinline__ float dot8_bf16(const bf16x8& a, const bf16x8& b, float c) {
  c = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 0, 1), __builtin_shufflevector(b, b, 0, 1), c, false);
  c = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 2, 3), __builtin_shufflevector(b, b, 2, 3), c, false);
  c = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 4, 5), __builtin_shufflevector(b, b, 4, 5), c, false);
  c = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(a, a, 6, 7), __builtin_shufflevector(b, b, 6, 7), c, false);
  return c;
}

__device__ __forceinline__ bf16x4 pack4(float a0, float a1, float a2, float a3) {
  bf16x4 r;
  r[0] = (bf16)a0; r[1] = (bf16)a1; r[2] = (bf16)a2; r[3] = (bf16)a3;
  return r;
}

__device__ __forceinline__ float xor32(float x) { return __shfl_xor(x, 32); }

// ds_read_b64_tr_b16: inside every group of 16 lanes, lane i receives element
// i%4 of the 8-byte chunks addressed by lanes 4e + i/4 (e = 0..3).  If lane j
// addresses row k0 + j/4, column n0 + 4*(j%4) of a row-major tile T[k][n],
// lane i therefore receives the column T[k0+e][n0+i], e = 0..3.
typedef short s16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ bf16x4 ld_tr4(const bf16* p) {
  const s16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(p));
  return __builtin_bit_cast(bf16x4, r);
}

// Direct global -> LDS copy (global_load_lds_dwordx4): lane i of the
// wavefront reads 16 bytes at `src` and the hardware writes them to
// lds_base + 16*i; lds_base must be the same for every lane.  Completion is
// tracked by the vector-memory counter.
__device__ __forceinline__ void dma16(const void* src, void* lds_base) {
  __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)(lds_base), 16, 0, 0);
}

// LDS tiles of R rows x 128 bf16 columns (one head) are stored as four
// 32-column planes, plane-major: plane p holds columns 32p..32p+31 of every
// row, 64 bytes per row, and the four 16-byte chunks of row r inside a plane
// are XOR-permuted by (r/4)%4.  With 64 LDS banks (256 bytes per cycle):
//  * 16-byte row reads (MFMA operands, 16 lanes = 16 aligned rows at one
//    column chunk) hit bank group 4*(r%4) + (chunk ^ (r/4)%4): 16 distinct;
//  * 8-byte transposed reads (ds_read_b64_tr_b16, 32 lanes = 4 aligned rows
//    x 32 columns of one plane) cover 256 contiguous bytes;
//  * a direct global-to-LDS load (64 lanes x 16 bytes, contiguous) fills 16
//    rows of one plane.
// Moving to another plane, or to rows 16 further down, only adds a constant
// to the address, so one base register serves many reads.
template <int R>
__device__ __forceinline__ int tile_off(int r, int c) {
  return (((c >> 5) * R + r) << 5) + (((((c >> 3) & 3) ^ ((r >> 2) & 3))) << 3) + (c & 7);
}

// MFMA operand (8 reduction values per lane) read column-wise from a plane
// tile T[k][n] of R rows: lane l takes column n0 + l%32 (n0 a multiple of 32);
// its reduction slots 0..3 come from rows ka..ka+3 and slots 4..7 from rows
// kb..kb+3 (ka, kb multiples of 4; they may depend on the lane's half l/32).
template <int R>
__device__ __forceinline__ bf16x8 ld_tr8(const bf16* T, int n0, int ka, int kb, int lane) {
  const int i = lane & 15;
  const int col = n0 + (lane & 16) + 4 * (i & 3);
  const bf16x4 lo = ld_tr4(T + tile_off<R>(ka + (i >> 2), col));
  const bf16x4 hi = ld_tr4(T + tile_off<R>(kb + (i >> 2), col));
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Direct load of rows into a plane tile of R rows: instruction m of a
// fetch (m = 0 .. R/4 - 1) fills rows 16*(m/4).. of plane m%4; lane i of it
// carries row 16*(m/4) + i/4 and the logical 8-column chunk returned by
// dma_col.  The caller supplies the row's global address.
template <int R>
__device__ __forceinline__ int dma_row(int m, int lane) { return 16 * (m >> 2) + (lane >> 2); }
template <int R>
__device__ __forceinline__ int dma_col(int m, int lane) {
  const int row = dma_row<R>(m, lane);
  return 32 * (m & 3) + 8 * ((lane & 3) ^ ((row >> 2) & 3));
}
template <int R>
__device__ __forceinline__ bf16* dma_dst(bf16* T, int m) {
  return T + (((m & 3) * R + 16 * (m >> 2)) << 5);
}
// the same destination as a byte offset from the tile's start
template <int R>
__device__ __forceinline__ constexpr uint32_t dma_dst_bytes(int m) {
  return (uint32_t)((((m & 3) * R + 16 * (m >> 2)) << 5) * 2);
}

// The same copies issued as inline assembly, invisible to the compiler's
// wait-count tracking.  The builtin above makes the compiler wait for every
// outstanding direct load before any LDS read it cannot prove disjoint,
// which serialises a prefetch pipeline; with these the caller waits on the
// vector-memory counter itself (wait_vmcnt) before the data is read.  Any
// compiler-visible vector-memory access (a global load, a register spill)
// issued while such loads are in flight makes the compiler's own waits
// cover them too, so loops that use these must be free of both.
// The address is a wavefront-uniform base plus a 32-bit per-lane byte
// offset; m0 carries the LDS base, also wavefront-uniform.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ const void* uniform_ptr(const void* p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (const void*)(uintptr_t)(((uint64_t)hi << 32) | lo);
}
// (a direct load reads M0 one wait state after a scalar write of it at the
// earliest: the s_nop 0 between them is that wait state)
__device__ __forceinline__ void dma16_async(const void* base, uint32_t off, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base),
               "s"(__builtin_amdgcn_readfirstlane(lds_addr))
               : "memory", "m0");
}
__device__ __forceinline__ void dma4_async(const void* base, uint32_t off, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1" ::"v"(off), "s"(base),
               "s"(__builtin_amdgcn_readfirstlane(lds_addr))
               : "memory", "m0");
}
#pragma clang diagnostic pop

// 32-bit LDS address of a shared-memory pointer, as a wavefront-uniform
// value.  Take it once per kernel and add byte offsets: converting generic
// pointers inside a loop costs a null check and 64-bit registers.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)(p));
}
// Per-lane LDS byte address, and 16-byte / transposed 8-byte reads at such
// an address: a compile-time constant added to the address folds into the
// instruction's offset field, so fragments at fixed distances from one base
// cost no address arithmetic.
__device__ __forceinline__ uint32_t lds_lane_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)(p);
}
__device__ __forceinline__ bf16x8 lds_ld16(uint32_t a) {
  return *(const __attribute__((address_space(3))) bf16x8*)(uintptr_t)a;
}
__device__ __forceinline__ bf16x4 lds_ld8(uint32_t a) {
  return *(const __attribute__((address_space(3))) bf16x4*)(uintptr_t)a;
}
__device__ __forceinline__ void lds_st16(uint32_t a, const bf16x8& v) {
  *(__attribute__((address_space(3))) bf16x8*)(uintptr_t)a = v;
}
__device__ __forceinline__ bf16x4 lds_ld_tr4(uint32_t a) {
  const s16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(uintptr_t)a);
  return __builtin_bit_cast(bf16x4, r);
}

// s_waitcnt vmcnt(N) (expcnt and lgkmcnt left alone) / vmcnt(N) lgkmcnt(0)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
template <int N>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

// Workgroup barrier that, unlike __syncthreads, does not drain the vector
// memory counter; the caller has already waited for what the other
// wavefronts will read.  The empty asm statements keep the compiler from
// moving memory accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Compile-time loop: f(std::integral_constant<int, i>) for i = 0 .. N-1, so
// that every index inside the body is a constant even where a large body
// would exceed the unroller's limits.
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int Ctrl>
__device__ __forceinline__ float dpp_mov(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), Ctrl, 0xF, 0xF, true));
}
// Sum over the 16 lanes of a DPP row (lanes 16r .. 16r+15); every lane of
// the row receives the sum.  All lanes of the wavefront must be active.
__device__ __forceinline__ float row16_sum(float x) {
  x += dpp_mov<0x128>(x);  // row_ror:8
  x += dpp_mov<0x124>(x);  // row_ror:4
  x += dpp_mov<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp_mov<0xB1>(x);   // quad_perm [1,0,3,2]
  return x;
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

}  // namespace ba
