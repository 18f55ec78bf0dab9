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

static unsigned rope_grid(int64_t rows) { return (unsigned)((rows * 16 + 255) / 256); }

hipError_t launch_rope_rows(const bf16* src, bf16* dst, const int32_t* pos, const RopeFreq* freq, int64_t rows,
                            int heads, hipStream_t stream) {
  if (rows <= 0) return hipSuccess;
  hipLaunchKernelGGL((rope_kernel<bf16, bf16, -1>), dim3(rope_grid(rows)), dim3(256), 0, stream, src, dst, pos,
                     freq, rows, heads, 1);
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
