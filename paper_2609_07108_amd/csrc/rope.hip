// Rotary position embedding of the branch-attention inputs and the
// transposed rotation of their gradients: the step in front of the op inside
// a draft layer.  Positions (the paper gives none for branch tokens): a main
// token at position p of its sequence has position p, member i of a branch
// group anchored at a has position a + 1 + i.  Dims j and j + 64 of a row
// turn together by the angle pos * theta^(-j/64).
//
// Memory-bound passes: one 16-lane DPP row per token row, looping over the
// row's heads (the angles are computed once per row and lane), a lane
// holding eight dims; the partner dims (j + 64 for j < 64 and back) sit in
// lane (l + 8) mod 16 of the same DPP row.  Rows whose position is negative
// are neither read nor written.
#include <type_traits>

#include "ba_internal.h"
#include "device_common.h"
#include "kernels.h"

namespace ba {
namespace {

constexpr int kRopeHeads = 4;  // heads loaded together, before any is used

__device__ __forceinline__ void load8(const bf16* p, float (&x)[8]) {
  const bf16x8 v = ld16(p);
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = (float)v[e];
}
__device__ __forceinline__ void load8(const float* p, float (&x)[8]) {
  const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
  x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
  x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}
__device__ __forceinline__ void store8(bf16* p, const float (&y)[8]) {
  st16(p, pack8(y[0], y[1], y[2], y[3], y[4], y[5], y[6], y[7]));
}
__device__ __forceinline__ void store8(float* p, const float (&y)[8]) {
  *reinterpret_cast<float4*>(p) = make_float4(y[0], y[1], y[2], y[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(y[4], y[5], y[6], y[7]);
}

}  // namespace

// dst[r, h] = R(pos[r]) src[r, h] (kSign = -1), or R(pos[r])^T src[r, h]
// (kSign = +1, the gradient direction), or a plain copy with conversion
// (rotate == 0); rows are [heads, 128].  Lanes l < 8 hold dims 8l..8l+7
// (the first of each pair): y = x cos + kSign x' sin; lanes l >= 8 hold the
// second: y = x cos - kSign x' sin, x' being the partner's value.
template <typename Src, typename Dst, int kSign>
__global__ __launch_bounds__(256) void rope_kernel(const Src* __restrict__ src, Dst* __restrict__ dst,
                                                   const int32_t* __restrict__ pos,
                                                   const RopeFreq* __restrict__ freq, int64_t rows, int heads,
                                                   int rotate) {
  const int lane = threadIdx.x & 63;
  const int64_t r0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4;
  const int64_t r = r0 < rows ? r0 : rows - 1;  // rows past the end redo the last row and write nothing
  const int ps = pos[r];
  const bool live = r0 < rows && ps >= 0;
  const int l = lane & 15;
  const float sg = l < 8 ? (float)kSign : (float)-kSign;
  float cs[8], sn[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    cs[e] = 1.f;
    sn[e] = 0.f;
  }
  if (rotate && ps >= 0) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      rope_sincos(ps, freq[8 * (l & 7) + e], sn[e], cs[e]);
      sn[e] *= sg;
    }
  }
  const int64_t base = r * heads * kHeadDim + 8 * l;
  for (int h0 = 0; h0 < heads; h0 += kRopeHeads) {
    float x[kRopeHeads][8];
#pragma unroll
    for (int u = 0; u < kRopeHeads; ++u) {
      const int h = h0 + u < heads ? h0 + u : h0;
      if (live) load8(src + base + (int64_t)h * kHeadDim, x[u]);
      else
#pragma unroll
        for (int e = 0; e < 8; ++e) x[u][e] = 0.f;
    }
    __builtin_amdgcn_sched_barrier(0);  // keep the loads together, ahead of their uses
#pragma unroll
    for (int u = 0; u < kRopeHeads; ++u) {
      float y[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float xp = dpp_mov<0x128>(x[u][e]);  // row_ror:8, the partner lane l ^ 8
        y[e] = fmaf(xp, sn[e], x[u][e] * cs[e]);
      }
      if (live && h0 + u < heads) store8(dst + base + (int64_t)(h0 + u) * kHeadDim, y);
    }
  }
}

// bf16 bits of v rounded to nearest, ties to even, in one step from double
// (no intermediate float rounding); values below bf16's normal range go
// through float (the rotated inputs never get there but for exact zeros).
__device__ __forceinline__ bf16 bf16_from_double(double v) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  const int be = (int)((b >> 52) & 0x7ff) - 1023 + 127;  // bf16 biased exponent
  if (be <= 0) return (bf16)(float)v;
  uint32_t r = ((uint32_t)be << 7) | (uint32_t)((b >> 45) & 0x7f);
  const uint64_t rest = b & ((1ull << 45) - 1), half = 1ull << 44;
  if (rest > half || (rest == half && (r & 1u))) ++r;  // a carry moves into the exponent
  r = r < 0x7f80u ? r : 0x7f80u;                       // past the largest finite: infinity
  return __builtin_bit_cast(bf16, (uint16_t)(((uint32_t)(b >> 48) & 0x8000u) | r));
}

// a double from lane l ^ 8 of the 16-lane DPP row (row_ror:8 on both halves)
__device__ __forceinline__ double dpp_ror8_f64(double x) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(x), 0x128, 0xF, 0xF, true);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(x), 0x128, 0xF, 0xF, true);
  return __hiloint2double(hi, lo);
}

// The rotation of the attention's bf16 inputs, R(pos) src (kSign = -1 of
// rope_kernel).  Angle pos * theta^(-j/64), its sine and cosine and the two
// products and their sum are each taken in double (no fused multiply-add),
// and the result is rounded once to bf16.  A float evaluation differs from
// the double one by a few float ulps, which moves about 3 in 10^5 values
// across a bf16 rounding midpoint; one such value on a key that dominates a
// short branch row shifts the row's LSE by about 1e-3, so the rounding is
// decided on the double value.  The stream is bound by HBM either way.
__global__ __launch_bounds__(256) void rope_in_kernel(const bf16* __restrict__ src, bf16* __restrict__ dst,
                                                      const int32_t* __restrict__ pos,
                                                      const double* __restrict__ rad, int64_t rows, int heads) {
#pragma clang fp contract(off)
  const int lane = threadIdx.x & 63;
  const int64_t r0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 4;
  const int64_t r = r0 < rows ? r0 : rows - 1;  // rows past the end redo the last row and write nothing
  const int ps = pos[r];
  const bool live = r0 < rows && ps >= 0;
  const int l = lane & 15;
  // lanes l < 8: y = x cos - x' sin (first dim of each pair); l >= 8: y = x cos + x' sin
  const double sg = l < 8 ? -1.0 : 1.0;
  // lanes l and l ^ 8 turn the same 8 pairs: each takes the sine and cosine
  // of 4 of the angles, and the partner's 4 come over by a DPP row rotation
  const int h4 = l < 8 ? 0 : 4;
  double so[4], co[4], sp[4], cp[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) sincos((double)(ps >= 0 ? ps : 0) * rad[8 * (l & 7) + h4 + k], &so[k], &co[k]);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    sp[k] = dpp_ror8_f64(so[k]);
    cp[k] = dpp_ror8_f64(co[k]);
  }
  double cs[8], sn[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const bool own = (e < 4) == (l < 8);
    cs[e] = own ? co[e & 3] : cp[e & 3];
    sn[e] = sg * (own ? so[e & 3] : sp[e & 3]);
  }
  const int64_t base = r * heads * kHeadDim + 8 * l;
  for (int h0 = 0; h0 < heads; h0 += kRopeHeads) {
    float x[kRopeHeads][8];
#pragma unroll
    for (int u = 0; u < kRopeHeads; ++u) {
      const int h = h0 + u < heads ? h0 + u : h0;
      if (live) load8(src + base + (int64_t)h * kHeadDim, x[u]);
      else
#pragma unroll
        for (int e = 0; e < 8; ++e) x[u][e] = 0.f;
    }
    __builtin_amdgcn_sched_barrier(0);  // keep the loads together, ahead of their uses
#pragma unroll
    for (int u = 0; u < kRopeHeads; ++u) {
      bf16x8 y;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float xp = dpp_mov<0x128>(x[u][e]);  // row_ror:8, the partner lane l ^ 8
        const double p0 = (double)x[u][e] * cs[e];
        const double p1 = (double)xp * sn[e];
        y[e] = bf16_from_double(p0 + p1);
      }
      if (live && h0 + u < heads) st16(dst + base + (int64_t)(h0 + u) * kHeadDim, y);
    }
  }
}

static unsigned rope_grid(int64_t rows) { return (unsigned)((rows * 16 + 255) / 256); }

hipError_t launch_rope_rows(const bf16* src, bf16* dst, const int32_t* pos, const double* rad, int64_t rows,
                            int heads, hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(rope_in_kernel, dim3(rope_grid(rows)), dim3(256), 0, stream, src, dst, pos, rad, rows, heads);
  return hipGetLastError();
}

hipError_t launch_rope_grad(const float* src, void* dst, bool dst_f32, const int32_t* pos, const RopeFreq* freq,
                            int64_t rows, int heads, bool rotate, hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  if (dst_f32)
    hipLaunchKernelGGL((rope_kernel<float, float, 1>), dim3(rope_grid(rows)), dim3(256), 0, stream, src,
                       static_cast<float*>(dst), pos, freq, rows, heads, rotate ? 1 : 0);
  else
    hipLaunchKernelGGL((rope_kernel<float, bf16, 1>), dim3(rope_grid(rows)), dim3(256), 0, stream, src,
                       static_cast<bf16*>(dst), pos, freq, rows, heads, rotate ? 1 : 0);
  return hipGetLastError();
}

}  // namespace ba
