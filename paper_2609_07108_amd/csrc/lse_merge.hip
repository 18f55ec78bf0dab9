// Standalone log-sum-exp merge of a partial attention result into a running
// one (Eq. lse-merge).  HBM-bound: each (row, head) pair reads its two LSEs
// and both outputs once and writes the merged output once.
#include "ba_internal.h"
#include "device_common.h"

namespace ba {

// A group of 32 lanes (half a wavefront) handles one (row, head) pair and
// walks its float4 chunks; every lane reads both LSEs before lane 0 of the
// group overwrites the running one, which keeps the in-place update race-free.
template <bool kPartBf16>
__global__ __launch_bounds__(256) void lse_merge_kernel(int64_t rows, int32_t heads, int32_t head_dim,
                                                        float* __restrict__ o_acc,
                                                        float* __restrict__ lse_acc,
                                                        const void* __restrict__ o_part,
                                                        const float* __restrict__ lse_part) {
  const int32_t q = head_dim / 4;
  const int64_t npairs = rows * heads;
  const int32_t sub = threadIdx.x & 31;
  for (int64_t pair = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 5; pair < npairs;
       pair += ((int64_t)gridDim.x * blockDim.x) >> 5) {
    const int64_t row = pair / heads;
    const int32_t head = (int32_t)(pair - row * heads);
    const int64_t li = (int64_t)head * rows + row;
    const float la = lse_acc[li];
    const float lb = lse_part[li];
    const float hi = fmaxf(la, lb);
    float wa = 0.f, wb = 0.f, l = -INFINITY;
    if (hi != -INFINITY) {
      const float ea = la == -INFINITY ? 0.f : expf(la - hi);
      const float eb = lb == -INFINITY ? 0.f : expf(lb - hi);
      const float tot = ea + eb;
      l = hi + logf(tot);
      wa = ea / tot;
      wb = eb / tot;
    }
    for (int32_t part = sub; part < q; part += 32) {
      float4* oa = reinterpret_cast<float4*>(o_acc + pair * head_dim) + part;
      float4 a = *oa;
      float4 b;
      if (kPartBf16) {
        const bf16x4 v =
            reinterpret_cast<const bf16x4*>(static_cast<const bf16*>(o_part) + pair * head_dim)[part];
        b = make_float4((float)v[0], (float)v[1], (float)v[2], (float)v[3]);
      } else {
        b = reinterpret_cast<const float4*>(static_cast<const float*>(o_part) + pair * head_dim)[part];
      }
      float4 o;
      o.x = wa * a.x + wb * b.x;
      o.y = wa * a.y + wb * b.y;
      o.z = wa * a.z + wb * b.z;
      o.w = wa * a.w + wb * b.w;
      *oa = o;
    }
    if (sub == 0) lse_acc[li] = l;
  }
}

}  // namespace ba

extern "C" int lse_merge(void* stream, int64_t rows, int32_t heads, int32_t head_dim, float* o_acc,
                         float* lse_acc, const void* o_part, int32_t o_part_dtype,
                         const float* lse_part) {
  if (rows < 0 || heads < 1 || head_dim < 4 || head_dim % 4 != 0) {
    ba::set_error("lse_merge: need rows >= 0, heads >= 1 and head_dim a positive multiple of 4");
    return BA_E_INVAL;
  }
  if (o_part_dtype != BA_DTYPE_BF16 && o_part_dtype != BA_DTYPE_F32) {
    ba::set_error("lse_merge: o_part_dtype must be BA_DTYPE_BF16 or BA_DTYPE_F32");
    return BA_E_INVAL;
  }
  if (rows == 0) return BA_OK;
  if (!o_acc || !lse_acc || !o_part || !lse_part) {
    ba::set_error("lse_merge: NULL pointer");
    return BA_E_INVAL;
  }
  const size_t align = o_part_dtype == BA_DTYPE_BF16 ? 8 : 16;
  if (((uintptr_t)o_acc & 15) || ((uintptr_t)o_part & (align - 1))) {
    ba::set_error("lse_merge: o_acc must be 16-byte and o_part element-vector aligned");
    return BA_E_INVAL;
  }
  const int64_t total = rows * heads * 32;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (o_part_dtype == BA_DTYPE_BF16)
    hipLaunchKernelGGL(ba::lse_merge_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, s, rows, heads,
                       head_dim, o_acc, lse_acc, o_part, lse_part);
  else
    hipLaunchKernelGGL(ba::lse_merge_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, s, rows, heads,
                       head_dim, o_acc, lse_acc, o_part, lse_part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    ba::set_error(std::string("lse_merge launch: ") + hipGetErrorString(e));
    return BA_E_HIP;
  }
  return BA_OK;
}
