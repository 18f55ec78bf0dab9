// Kernel parameter blocks and launchers (device side of the library).
#pragma once
#include <hip/hip_runtime.h>

#include "ba_internal.h"
#include "device_common.h"

namespace ba {

constexpr int kMaxCp = 32;  // ring steps whose block pointers fit in a kernel argument

constexpr int kModeStep = 0;   // one ring step, merge into the running pair
constexpr int kModeFinal = 1;  // branch-local part + merge + write, main part from the running pair
constexpr int kModeFused = 2;  // every ring step + branch-local part + merge + write

struct FwdParams {
  const SeqInfo* seqs;
  const TokInfo* toks;
  const GroupInfo* groups;
  const FwdTile* tiles;
  int32_t num_tiles;
  int32_t C, rank, hq, hkv, G;
  float scale_log2;  // softmax scale * log2(e)
  int64_t n_local;
  int64_t n_br;
  const bf16* q_main;
  const bf16* q_br;
  const bf16* k_br;
  const bf16* v_br;
  const bf16* k_step[kMaxCp];
  const bf16* v_step[kMaxCp];
  bf16* o_main;
  bf16* o_br;
  float* lse_main;
  float* lse_br;
  float* o_acc;    // [T * hq, d] running output (per-step schedule)
  float* lse_acc;  // [T * hq] running LSE, log2 units
  int32_t step_first, step_count, acc_first;
};

struct BwdParams {
  const SeqInfo* seqs;
  const TokInfo* toks;
  const GroupInfo* groups;
  const BwdTile* tiles;   // key tiles of the dK/dV kernel
  int32_t num_tiles;
  const FwdTile* qtiles;  // query tiles of the dQ kernel
  int32_t num_qtiles;
  int32_t step_first, step_count, acc_first;
  int32_t C, rank, hq, hkv, G;
  int32_t num_tokens;
  int32_t num_groups;
  float scale;       // softmax scale
  float scale_log2;  // softmax scale * log2(e)
  int64_t n_local;
  int64_t n_br;
  const bf16* q_main;
  const bf16* q_br;
  const bf16* k_br;
  const bf16* v_br;
  const bf16* k_step[kMaxCp];
  const bf16* v_step[kMaxCp];
  const bf16* o_main;
  const bf16* o_br;
  const float* lse_main;
  const float* lse_br;
  const bf16* do_main;
  const bf16* do_br;
  void* dq_main;
  void* dq_br;
  void* dk_step[kMaxCp];
  void* dv_step[kMaxCp];
  void* dk_br;
  void* dv_br;
  int32_t grad_f32;
  float2* rowstat;  // [T * hq]: (-LSE * log2 e, -Delta = -<dO, O>)
  bf16* qtok;       // [T * hq, d] Q rows in token order (written by the preprocess)
  bf16* gtok;       // [T * hq, d] dO rows in token order
  float* dq_acc;    // [T * hq, d] running unscaled dS K sums (per-step schedule)
};

// Walk over the 64-key tiles of every ring step in [step_first,
// step_first + step_count) that a query tile with largest causal limit Pmax
// can see.  Each tile's K and V rows are fetched with direct global-to-LDS
// loads into plane tiles (see tile_off), double-buffered: while `body`
// computes on one buffer the next tile, possibly of the next ring step, is
// already in flight into the other.  The loads are not tracked by the
// compiler (dma16_async), so the body's LDS reads do not wait for them; the
// walk waits explicitly before each barrier, and the body issues no global
// loads of its own.  The buffers are used in a fixed
// alternation so their LDS addresses are compile-time constants in the body.
// body(j, kv0, ks, vs) is called once per tile with the ring block j, the
// first key kv0 (index inside the sequence's segment of block j) and the
// staged K and V tiles; rows past the block's visible prefix hold clamped
// copies and must be masked by the body.
struct KvCursor {
  int i, j, kv0, lim_hi;
};

template <class P, class Body>
__device__ __forceinline__ void walk_kv_tiles(const P& p, const SeqInfo& seq, int kvh, int Pmax, int wave,
                                              int lane, bf16 (&kv)[2][2][kFwdKeys * kHeadDim], Body&& body) {
  const int step_end = p.step_first + p.step_count;
  const int64_t stride = (int64_t)p.hkv * kHeadDim;
  auto seek = [&](int i) {
    KvCursor c{i, 0, 0, 0};
    for (; c.i < step_end; ++c.i) {
      c.j = ((p.rank - c.i) % p.C + p.C) % p.C;  // ring step i brings rank (r - i) mod C
      c.lim_hi = visible_keys(Pmax, c.j, p.C, seq.c);
      if (c.lim_hi > 0) break;
    }
    return c;
  };
  auto next = [&](KvCursor c) {
    c.kv0 += kFwdKeys;
    return c.kv0 < c.lim_hi ? c : seek(c.i + 1);
  };
  constexpr uint32_t kTileBytes = kFwdKeys * kHeadDim * sizeof(bf16);
  const uint32_t kv_lds = lds_addr(&kv[0][0][0]);  // [buffer][K, V] tiles follow each other
  auto fetch = [&](const KvCursor& c, int buf) {
    const uint32_t kd = kv_lds + (2 * buf) * kTileBytes, vd = kd + kTileBytes;
    // base: the tile's first key row (uniform); per lane a byte offset
    const int64_t row0 = ((int64_t)seq.seg_off + c.kv0) * stride + kvh * kHeadDim;
    const void* kb = uniform_ptr(p.k_step[c.j] + row0);
    const void* vb = uniform_ptr(p.v_step[c.j] + row0);
    const int nrow = c.lim_hi - c.kv0;  // rows past the visible prefix repeat its last row
#pragma unroll
    for (int m4 = 0; m4 < 4; ++m4) {
      const int m = 4 * wave + m4;  // 16 loads per tensor and tile, 4 per wavefront
      int u = dma_row<kFwdKeys>(m, lane);
      u = u < nrow ? u : nrow - 1;
      const uint32_t off = (uint32_t)(u * (int)stride + dma_col<kFwdKeys>(m, lane)) * (uint32_t)sizeof(bf16);
      dma16_async(kb, off, kd + dma_dst_bytes<kFwdKeys>(m));
      dma16_async(vb, off, vd + dma_dst_bytes<kFwdKeys>(m));
    }
  };
  KvCursor cur = seek(p.step_first);
  if (cur.i >= step_end) return;
  fetch(cur, 0);
  __builtin_amdgcn_s_waitcnt(0);
  lds_barrier();
  while (true) {
    KvCursor nx = next(cur);
    if (nx.i < step_end) fetch(nx, 1);
    body(cur.j, cur.kv0, kv[0][0], kv[0][1]);
    wait_vmcnt_lgkm0<0>();  // this wavefront's loads of the next tile have landed
    lds_barrier();
    if (nx.i >= step_end) return;
    cur = nx;
    nx = next(cur);
    if (nx.i < step_end) fetch(nx, 0);
    body(cur.j, cur.kv0, kv[1][0], kv[1][1]);
    wait_vmcnt_lgkm0<0>();
    lds_barrier();
    if (nx.i >= step_end) return;
    cur = nx;
  }
}

hipError_t launch_fwd(const FwdParams& p, int mode, hipStream_t stream);
hipError_t launch_bwd_preprocess(const BwdParams& p, hipStream_t stream);
hipError_t launch_bwd_kv(const BwdParams& p, hipStream_t stream);
hipError_t launch_bwd_dq(const BwdParams& p, int mode, hipStream_t stream);
hipError_t launch_bwd_branch(const BwdParams& p, int max_group_len, hipStream_t stream);
hipError_t launch_zero(void* ptr, size_t bytes, hipStream_t stream);

}  // namespace ba
