// Backward branch attention for one context-parallel rank share (Sec. 3.2:
// the backward pass replays the same KV ring and accumulates gradients
// locally).
//
// Using the final LSE of every row, the probabilities of any key set are
// P = exp(S - LSE), and the merge of Eq. lse-merge needs no explicit
// backward: each ring-step block and the branch-local keys contribute
//   dV += P^T dO,  dS = P o (dP - Delta) with dP = dO V^T and
//   Delta = <dO, O>,  dK += scale dS^T Q,  dQ += scale dS K.
//
// Kernels
//   preprocess : Delta and LSE * log2(e) per (token, head); clears dQ sums.
//   main       : one workgroup per 128 keys of one ring-step block, one
//                sequence and one KV head (32 keys per wavefront, dK and dV in
//                registers).  It walks the query tokens that see those keys in
//                64-row tiles (tokens x the G heads of the KV head); dQ
//                contributions are summed over the 128 keys through LDS and
//                added to an fp32 accumulator with global atomics.
//   branch     : branch-local keys (at most 64 per group), vector ALUs.
//   finalize   : dQ = scale * sums, converted to the output dtype.
#include "ba_internal.h"
#include "device_common.h"
#include "kernels.h"

namespace ba {

namespace {

constexpr int kRowStride = kHeadDim + 8;  // padded row-major [rows][d] tiles
constexpr int kKtStride = kBwdKeys + 8;   // K^T tile [d][keys]
constexpr int kDsStride = kBwdKeys + 8;   // dS tile [rows][keys]

// Transposed [d][64 rows] tile whose 16-byte chunk 2t+h holds rows
// 16t+4h+{0..3} then 16t+8+4h+{0..3}, the rows a lane of half h feeds into
// k-block t of an MFMA from an accumulator.  XOR-swizzled per d.
__device__ __forceinline__ int tr_index(int d, int lchunk) {
  const int sw = (d ^ (d >> 3)) & 7;
  return d * kBwdRows + ((lchunk ^ sw) << 3);
}

__device__ __forceinline__ const bf16* row_ptr(const bf16* main, const bf16* br, int32_t qrow,
                                               int32_t hq, int32_t head) {
  return qrow >= 0 ? main + ((int64_t)qrow * hq + head) * kHeadDim
                   : br + ((int64_t)(-qrow - 1) * hq + head) * kHeadDim;
}

__device__ __forceinline__ void store_grad(void* base, int64_t idx, float v, bool f32) {
  if (f32) static_cast<float*>(base)[idx] = v;
  else static_cast<bf16*>(base)[idx] = (bf16)v;
}

}  // namespace

// ------------------------------------------------------------ preprocess
// 32 lanes per (token, head): Delta = <dO, O> over 128 dims, the row's LSE in
// log2 units, and a cleared dQ accumulator row.
__global__ __launch_bounds__(256) void bwd_preprocess_kernel(BwdParams p) {
  const int64_t pair = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 5;
  const int sub = threadIdx.x & 31;
  if (pair >= (int64_t)p.num_tokens * p.hq) return;
  const int32_t t = (int32_t)(pair / p.hq);
  const int32_t head = (int32_t)(pair - (int64_t)t * p.hq);
  const TokInfo tk = p.toks[t];
  const bf16* o = row_ptr(p.o_main, p.o_br, tk.qrow, p.hq, head);
  const bf16* g = row_ptr(p.do_main, p.do_br, tk.qrow, p.hq, head);
  const bf16x4 ov = reinterpret_cast<const bf16x4*>(o)[sub];
  const bf16x4 gv = reinterpret_cast<const bf16x4*>(g)[sub];
  float dlt = (float)ov[0] * (float)gv[0] + (float)ov[1] * (float)gv[1] + (float)ov[2] * (float)gv[2] +
              (float)ov[3] * (float)gv[3];
#pragma unroll
  for (int m = 16; m >= 1; m >>= 1) dlt += __shfl_xor(dlt, m, 32);
  reinterpret_cast<float4*>(p.dq_acc + pair * kHeadDim)[sub] = make_float4(0.f, 0.f, 0.f, 0.f);
  if (sub == 0) {
    const float lse = tk.qrow >= 0 ? p.lse_main[(int64_t)head * p.n_local + tk.qrow]
                                   : p.lse_br[(int64_t)head * p.n_br + (-tk.qrow - 1)];
    p.rowstat[pair] = make_float2(lse * kLog2e, dlt);
  }
}

// ------------------------------------------------------------ main (ring)
__global__ __launch_bounds__(256, 1) void bwd_main_kernel(BwdParams p) {
  __shared__ __attribute__((aligned(16))) bf16 q_s[kBwdRows * kRowStride];
  __shared__ __attribute__((aligned(16))) bf16 do_s[kBwdRows * kRowStride];
  __shared__ __attribute__((aligned(16))) bf16 qt_s[kHeadDim * kBwdRows];
  __shared__ __attribute__((aligned(16))) bf16 dot_s[kHeadDim * kBwdRows];
  __shared__ __attribute__((aligned(16))) bf16 ds_s[kBwdRows * kDsStride];
  __shared__ __attribute__((aligned(16))) bf16 kt_s[kHeadDim * kKtStride];
  __shared__ __attribute__((aligned(16))) float lse_s[kBwdRows];
  __shared__ __attribute__((aligned(16))) float dlt_s[kBwdRows];
  __shared__ __attribute__((aligned(16))) int lim_s[kBwdRows];

  const BwdTile tile = p.tiles[blockIdx.x];
  const SeqInfo seq = p.seqs[tile.seq];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int qi = lane & 31;
  const int half = lane >> 5;
  const int64_t kv_row_stride = (int64_t)p.hkv * kHeadDim;
  const int64_t key0 = (int64_t)seq.seg_off + tile.u0;  // first key row in the block
  const bf16* kbase = p.k_step[tile.step] + key0 * kv_row_stride + tile.kvh * kHeadDim;
  const bf16* vbase = p.v_step[tile.step] + key0 * kv_row_stride + tile.kvh * kHeadDim;

  // this lane's key (B operand of S = Q K^T and dP = dO V^T): key 32*wave+qi
  const int my_key = 32 * wave + qi;
  const int kload = my_key < tile.nk ? my_key : tile.nk - 1;
  bf16x8 kreg[8], vreg[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    kreg[c] = ld16(kbase + (int64_t)kload * kv_row_stride + 16 * c + 8 * half);
    vreg[c] = ld16(vbase + (int64_t)kload * kv_row_stride + 16 * c + 8 * half);
  }
  // K^T tile for dQ = dS K: kt_s[d][key]
  {
    const int kg = tid >> 3, dc = tid & 7;  // keys 4kg..4kg+3, dims 16dc..16dc+15
    bf16x8 kv[4][2];
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      int u = 4 * kg + r4;
      u = u < tile.nk ? u : tile.nk - 1;
      kv[r4][0] = ld16(kbase + (int64_t)u * kv_row_stride + 16 * dc);
      kv[r4][1] = ld16(kbase + (int64_t)u * kv_row_stride + 16 * dc + 8);
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      bf16x4 w;
      w[0] = kv[0][e >> 3][e & 7]; w[1] = kv[1][e >> 3][e & 7];
      w[2] = kv[2][e >> 3][e & 7]; w[3] = kv[3][e >> 3][e & 7];
      *reinterpret_cast<bf16x4*>(&kt_s[(16 * dc + e) * kKtStride + 4 * kg]) = w;
    }
  }

  f32x16 dk[4], dv[4];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt) {
    dk[nt] = f32x16{};
    dv[nt] = f32x16{};
  }

  const int G = p.G;
  const int tpt = kBwdRows / G;  // tokens per query tile
  for (int qt0 = tile.q_begin; qt0 < tile.q_end; qt0 += tpt) {
    __syncthreads();  // previous tile's LDS reads are done (and kt_s is written)
    // ---- stage Q, dO (row-major and transposed) and the row statistics
    {
      const int rg = tid >> 4, dc = tid & 15;  // rows 4rg..4rg+3, dims 8dc..8dc+7
      bf16x8 qv[4], gv[4];
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int r = 4 * rg + r4;
        const int tl = r / G;
        const int tok = qt0 + tl;
        if (tok < tile.q_end) {
          const TokInfo tk = p.toks[tok];
          const int head = tile.kvh * G + (r - tl * G);
          qv[r4] = ld16(row_ptr(p.q_main, p.q_br, tk.qrow, p.hq, head) + 8 * dc);
          gv[r4] = ld16(row_ptr(p.do_main, p.do_br, tk.qrow, p.hq, head) + 8 * dc);
        } else {
          qv[r4] = bf16x8{};
          gv[r4] = bf16x8{};
        }
        st16(&q_s[r * kRowStride + 8 * dc], qv[r4]);
        st16(&do_s[r * kRowStride + 8 * dc], gv[r4]);
      }
      const int tb = rg >> 2, a = (rg & 3) >> 1, b = rg & 1;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = 8 * dc + e;
        bf16x4 w;
        w[0] = qv[0][e]; w[1] = qv[1][e]; w[2] = qv[2][e]; w[3] = qv[3][e];
        *reinterpret_cast<bf16x4*>(&qt_s[tr_index(d, 2 * tb + b) + 4 * a]) = w;
        w[0] = gv[0][e]; w[1] = gv[1][e]; w[2] = gv[2][e]; w[3] = gv[3][e];
        *reinterpret_cast<bf16x4*>(&dot_s[tr_index(d, 2 * tb + b) + 4 * a]) = w;
      }
    }
    if (tid < kBwdRows) {
      const int r = tid;
      const int tl = r / G;
      const int tok = qt0 + tl;
      float l2 = 0.f, dl = 0.f;
      int lim = 0;
      if (tok < tile.q_end) {
        const int head = tile.kvh * G + (r - tl * G);
        const float2 rs = p.rowstat[(int64_t)tok * p.hq + head];
        l2 = rs.x;
        dl = rs.y;
        lim = visible_keys(p.toks[tok].P, tile.step, p.C, seq.c) - tile.u0;
        lim = lim < tile.nk ? lim : tile.nk;
      }
      lse_s[r] = l2;
      dlt_s[r] = dl;
      lim_s[r] = lim;
    }
    __syncthreads();
    const bool need_mask = qt0 < tile.q_full || qt0 + tpt > tile.q_end || tile.nk < kBwdKeys;

    // ---- S = Q K^T and dP = dO V^T (rows = queries, columns = this lane's key)
    f32x16 s[2], dp[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      s[mt] = f32x16{};
      dp[mt] = f32x16{};
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        s[mt] = mfma32(ld16(&q_s[(32 * mt + qi) * kRowStride + 16 * c + 8 * half]), kreg[c], s[mt]);
        dp[mt] = mfma32(ld16(&do_s[(32 * mt + qi) * kRowStride + 16 * c + 8 * half]), vreg[c], dp[mt]);
      }
    }
    // ---- P = exp2(S scale log2e - LSE log2e), dS = P (dP - Delta)
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int vq = 0; vq < 4; ++vq) {
        const int r0 = 32 * mt + 8 * vq + 4 * half;
        const float4 l4 = *reinterpret_cast<const float4*>(&lse_s[r0]);
        const float4 d4 = *reinterpret_cast<const float4*>(&dlt_s[r0]);
        const int4 m4 = *reinterpret_cast<const int4*>(&lim_s[r0]);
        const float lr[4] = {l4.x, l4.y, l4.z, l4.w};
        const float dr[4] = {d4.x, d4.y, d4.z, d4.w};
        const int mr[4] = {m4.x, m4.y, m4.z, m4.w};
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int v = 4 * vq + c;
          float pr = fast_exp2(s[mt][v] * p.scale_log2 - lr[c]);
          if (need_mask && my_key >= mr[c]) pr = 0.f;
          s[mt][v] = pr;
          dp[mt][v] = pr * (dp[mt][v] - dr[c]);
        }
      }
    }
    // ---- dV += P^T dO, dK += dS^T Q (k-block t = query rows 16t..16t+15)
    bf16x8 pa[4], dsa[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int v0 = 8 * (t & 1);
      const f32x16& ps = s[t >> 1];
      const f32x16& dss = dp[t >> 1];
      pa[t] = pack8(ps[v0], ps[v0 + 1], ps[v0 + 2], ps[v0 + 3], ps[v0 + 4], ps[v0 + 5], ps[v0 + 6], ps[v0 + 7]);
      dsa[t] = pack8(dss[v0], dss[v0 + 1], dss[v0 + 2], dss[v0 + 3], dss[v0 + 4], dss[v0 + 5], dss[v0 + 6],
                     dss[v0 + 7]);
    }
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        dv[nt] = mfma32(pa[t], ld16(&dot_s[tr_index(32 * nt + qi, 2 * t + half)]), dv[nt]);
        dk[nt] = mfma32(dsa[t], ld16(&qt_s[tr_index(32 * nt + qi, 2 * t + half)]), dk[nt]);
      }
    }
    // ---- dS (bf16) to LDS as [row][key] for dQ = dS K
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = 32 * mt + 8 * (v >> 2) + 4 * half + (v & 3);
        ds_s[r * kDsStride + my_key] = (bf16)dp[mt][v];
      }
    __syncthreads();
    // ---- dQ tile (64 rows x 128 dims): wave w takes rows 32*(w&1).., dims 64*(w>>1)..
    {
      const int mt = wave & 1;
      f32x16 dq[2];
      dq[0] = f32x16{};
      dq[1] = f32x16{};
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const bf16x8 a = ld16(&ds_s[(32 * mt + qi) * kDsStride + 16 * c + 8 * half]);
#pragma unroll
        for (int n = 0; n < 2; ++n) {
          const int nt = 2 * (wave >> 1) + n;
          dq[n] = mfma32(a, ld16(&kt_s[(32 * nt + qi) * kKtStride + 16 * c + 8 * half]), dq[n]);
        }
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = 32 * mt + 8 * (v >> 2) + 4 * half + (v & 3);
        const int tl = r / G;
        const int tok = qt0 + tl;
        if (tok < tile.q_end) {
          const int head = tile.kvh * G + (r - tl * G);
          float* dst = p.dq_acc + ((int64_t)tok * p.hq + head) * kHeadDim;
#pragma unroll
          for (int n = 0; n < 2; ++n) atomicAdd(dst + 32 * (2 * (wave >> 1) + n) + qi, dq[n][v]);
        }
      }
    }
  }

  // ---- write dK (scaled) and dV of this lane's... C layout: column = d, rows = keys
  void* dkout = p.dk_step[tile.step];
  void* dvout = p.dv_step[tile.step];
#pragma unroll
  for (int nt = 0; nt < 4; ++nt)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int key = 32 * wave + 8 * (v >> 2) + 4 * half + (v & 3);
      if (key < tile.nk) {
        const int64_t idx = (key0 + key) * kv_row_stride + tile.kvh * kHeadDim + 32 * nt + qi;
        store_grad(dkout, idx, dk[nt][v] * p.scale, p.grad_f32);
        store_grad(dvout, idx, dv[nt][v], p.grad_f32);
      }
    }
}

// ------------------------------------------------------------ branch-local
// One workgroup per (group, KV head).  Each wavefront takes query rows
// (member i, head) in turn; lanes hold two dims each.  Scores and dP need a
// wavefront-wide reduction per key.  dK/dV of the group's keys are summed in
// LDS (fp32) and written once; a dQ row is owned by one wavefront and updated
// in place (the ring kernel has finished with it).
__global__ __launch_bounds__(256) void bwd_branch_kernel(BwdParams p) {
  extern __shared__ float acc_s[];  // [2][len][128]: dK sums, dV sums
  const int g = blockIdx.x / p.hkv;
  const int kvh = blockIdx.x - g * p.hkv;
  const GroupInfo gi = p.groups[g];
  const int n = gi.len;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int i = tid; i < 2 * n * kHeadDim; i += blockDim.x) acc_s[i] = 0.f;
  __syncthreads();
  const int64_t kv_row_stride = (int64_t)p.hkv * kHeadDim;
  const int G = p.G;
  for (int rr = wave; rr < n * G; rr += 4) {
    const int i = rr / G;
    const int head = kvh * G + (rr - i * G);
    const int64_t brow = (int64_t)gi.row0 + (int64_t)i * gi.stride;
    const bf16* q = p.q_br + (brow * p.hq + head) * kHeadDim;
    const bf16* g_ = p.do_br + (brow * p.hq + head) * kHeadDim;
    // row statistics: recomputed from O and the final LSE of this branch row
    const bf16* o = p.o_br + (brow * p.hq + head) * kHeadDim;
    const float q0 = (float)q[2 * lane], q1 = (float)q[2 * lane + 1];
    const float g0 = (float)g_[2 * lane], g1 = (float)g_[2 * lane + 1];
    float dlt = g0 * (float)o[2 * lane] + g1 * (float)o[2 * lane + 1];
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) dlt += __shfl_xor(dlt, m);
    const float lse2 = p.lse_br[(int64_t)head * p.n_br + brow] * kLog2e;
    const int nk = gi.kind == BA_KIND_EAGLE_CHAIN ? i + 1 : n;
    float dq0 = 0.f, dq1 = 0.f;
    for (int j = 0; j < nk; ++j) {
      const int64_t krow = (int64_t)gi.row0 + (int64_t)j * gi.stride;
      const bf16* kp = p.k_br + krow * kv_row_stride + kvh * kHeadDim;
      const bf16* vp = p.v_br + krow * kv_row_stride + kvh * kHeadDim;
      const float k0 = (float)kp[2 * lane], k1 = (float)kp[2 * lane + 1];
      const float v0 = (float)vp[2 * lane], v1 = (float)vp[2 * lane + 1];
      float sdot = q0 * k0 + q1 * k1;
      float pdot = g0 * v0 + g1 * v1;
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) {
        sdot += __shfl_xor(sdot, m);
        pdot += __shfl_xor(pdot, m);
      }
      const float pr = fast_exp2(sdot * p.scale_log2 - lse2);
      const float ds = pr * (pdot - dlt);
      dq0 += ds * k0;
      dq1 += ds * k1;
      atomicAdd(&acc_s[j * kHeadDim + 2 * lane], ds * q0);
      atomicAdd(&acc_s[j * kHeadDim + 2 * lane + 1], ds * q1);
      atomicAdd(&acc_s[(n + j) * kHeadDim + 2 * lane], pr * g0);
      atomicAdd(&acc_s[(n + j) * kHeadDim + 2 * lane + 1], pr * g1);
    }
    // group members are consecutive query tokens starting at gi.tok0
    float* dq = p.dq_acc + ((int64_t)(gi.tok0 + i) * p.hq + head) * kHeadDim;
    dq[2 * lane] += dq0;
    dq[2 * lane + 1] += dq1;
  }
  __syncthreads();
  for (int idx = tid; idx < n * kHeadDim; idx += blockDim.x) {
    const int j = idx / kHeadDim, d = idx - j * kHeadDim;
    const int64_t krow = (int64_t)gi.row0 + (int64_t)j * gi.stride;
    const int64_t o = krow * kv_row_stride + kvh * kHeadDim + d;
    store_grad(p.dk_br, o, acc_s[idx] * p.scale, p.grad_f32);
    store_grad(p.dv_br, o, acc_s[n * kHeadDim + idx], p.grad_f32);
  }
}

// ------------------------------------------------------------ finalize
// dQ = scale * (ring + branch-local sums), converted and scattered to the
// caller's layout.  One thread per 4 dims of a (token, head) row.
__global__ __launch_bounds__(256) void bwd_finalize_kernel(BwdParams p) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t pair = i >> 5;
  const int sub = (int)(i & 31);
  if (pair >= (int64_t)p.num_tokens * p.hq) return;
  const int32_t t = (int32_t)(pair / p.hq);
  const int32_t head = (int32_t)(pair - (int64_t)t * p.hq);
  const TokInfo tk = p.toks[t];
  float4 a = reinterpret_cast<const float4*>(p.dq_acc + pair * kHeadDim)[sub];
  a.x *= p.scale; a.y *= p.scale; a.z *= p.scale; a.w *= p.scale;
  void* out = tk.qrow >= 0 ? p.dq_main : p.dq_br;
  const int64_t row = tk.qrow >= 0 ? tk.qrow : -tk.qrow - 1;
  const int64_t base = (row * p.hq + head) * kHeadDim + 4 * sub;
  if (p.grad_f32) {
    *reinterpret_cast<float4*>(static_cast<float*>(out) + base) = a;
  } else {
    *reinterpret_cast<bf16x4*>(static_cast<bf16*>(out) + base) = pack4(a.x, a.y, a.z, a.w);
  }
}

__global__ __launch_bounds__(256) void zero_kernel(uint4* __restrict__ p, int64_t n16) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = make_uint4(0u, 0u, 0u, 0u);
}

static unsigned grid_for(int64_t threads) {
  int64_t b = (threads + 255) / 256;
  return (unsigned)(b < 1 ? 1 : b);
}

hipError_t launch_bwd_preprocess(const BwdParams& p, hipStream_t stream) {
  const int64_t threads = (int64_t)p.num_tokens * p.hq * 32;
  if (threads == 0) return hipSuccess;
  hipLaunchKernelGGL(bwd_preprocess_kernel, dim3(grid_for(threads)), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_bwd_main(const BwdParams& p, hipStream_t stream) {
  if (p.num_tiles == 0) return hipSuccess;
  hipLaunchKernelGGL(bwd_main_kernel, dim3(p.num_tiles), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_bwd_branch(const BwdParams& p, int max_group_len, hipStream_t stream) {
  if (p.num_groups == 0) return hipSuccess;
  const size_t lds = (size_t)2 * max_group_len * kHeadDim * sizeof(float);
  hipLaunchKernelGGL(bwd_branch_kernel, dim3(p.num_groups * p.hkv), dim3(256), lds, stream, p);
  return hipGetLastError();
}

hipError_t launch_bwd_finalize(const BwdParams& p, hipStream_t stream) {
  const int64_t threads = (int64_t)p.num_tokens * p.hq * 32;
  if (threads == 0) return hipSuccess;
  hipLaunchKernelGGL(bwd_finalize_kernel, dim3(grid_for(threads)), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_zero(void* ptr, size_t bytes, hipStream_t stream) {
  if (bytes == 0) return hipSuccess;
  const int64_t n16 = (int64_t)(bytes / 16);
  int64_t blocks = (n16 + 255) / 256;
  if (blocks > 16384) blocks = 16384;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(zero_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, static_cast<uint4*>(ptr), n16);
  return hipGetLastError();
}

}  // namespace ba
