// Kernel parameter blocks and launchers (device side of the library).
#pragma once
#include <hip/hip_runtime.h>

#include "ba_internal.h"
#include "device_common.h"

namespace ba {

constexpr int kMaxCp = 32;  // ring steps whose block pointers fit in a kernel argument

constexpr int kModeStep = 0;   // one ring step, merge into the running pair
constexpr int kModeFused = 2;  // every ring step + branch-local part + merge + write

struct FwdParams {
  const SeqInfo* seqs;
  const TokInfo* toks;
  const GroupInfo* groups;
  const FwdTile* tiles;
  int32_t num_tiles;
  const int32_t* br_keys;    // branch key rows of the tiles (FwdTile::bk_off)
  const int32_t* tok_bslot;  // per token: first slot of its group's keys in its tile
  int32_t C, rank, hq, hkv, G;
  int32_t num_tokens;
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
  const int32_t* br_keys;    // branch key rows of the query tiles (FwdTile::bk_off)
  const int32_t* tok_bslot;  // per token: first slot of its group's keys in its tile
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
  float* kv_part;   // [slots][dV, dK][kBwdKeys][d] partial sums of split work items
  const KvSplit* splits;
  int32_t num_splits;
};

// Cursor of a walk over (ring step i, block j = (rank - i) mod C, first key
// kv0 of a 64-key tile, keys of the block visible to the tile lim_hi).
struct KvCursor {
  int i, j, kv0, lim_hi;
  int lim_lo;  // keys of block j every row of the query tile sees (tiles below need no mask)
};

hipError_t launch_fwd(const FwdParams& p, int mode, hipStream_t stream);
hipError_t launch_fwd_finalize(const FwdParams& p, hipStream_t stream);
hipError_t launch_bwd_preprocess(const BwdParams& p, hipStream_t stream);
hipError_t launch_bwd_kv(const BwdParams& p, hipStream_t stream);
hipError_t launch_bwd_dq(const BwdParams& p, int mode, hipStream_t stream);
hipError_t launch_bwd_dq_finalize(const BwdParams& p, hipStream_t stream);
hipError_t launch_bwd_branch(const BwdParams& p, int max_group_len, hipStream_t stream);
hipError_t launch_bwd_kv_reduce(const BwdParams& p, hipStream_t stream);
hipError_t launch_zero(void* ptr, size_t bytes, hipStream_t stream);
// rotary embedding of bf16 rows [rows, heads, 128] (positions < 0: row
// skipped), evaluated in double from the radian table and rounded once
hipError_t launch_rope_rows(const bf16* src, bf16* dst, const int32_t* pos, const double* rad, int64_t rows,
                            int heads, hipStream_t stream);
// transposed rotation (or, with rotate false, a plain copy) of fp32 gradient
// rows into bf16 or fp32 rows
hipError_t launch_rope_grad(const float* src, void* dst, bool dst_f32, const int32_t* pos, const RopeFreq* freq,
                            int64_t rows, int heads, bool rotate, hipStream_t stream);


// Grouped-query QKV projection (proj.hip): C[i][j] = sum_k A(i,k) B(j,k) over
// 128 x 128 tiles.  An operand is stored k-major ([i][k], ld elements per
// row; its reduction slices must lie inside K) or i-major ([k][i]; its row
// count must be a multiple of 128, a ragged K is allowed).  J is a multiple
// of 128; I may be ragged where A is k-major.
constexpr int kProjEpiPlain = 0;  // C written row-major (ldc), bf16 or fp32, optionally added to
constexpr int kProjEpiQkv = 1;    // 128-column heads split into q / k / v, q and k rotated, bf16 THD

struct RopeFreqTable {
  RopeFreq f[kHeadDim / 2];
};

struct ProjGemmParams {
  const bf16* a;
  const bf16* b;
  int64_t lda, ldb;
  int64_t I, K;
  int32_t J;
  // plain epilogue
  int32_t c_f32, accumulate;
  void* c;
  int64_t ldc;
  // q / k / v epilogue
  bf16* q;
  bf16* k;
  bf16* v;
  int32_t hq, hkv, rotate;
  const int32_t* pos;
  RopeFreqTable freq;
};

hipError_t launch_proj_gemm(const ProjGemmParams& p, bool a_imajor, bool b_imajor, int epi, hipStream_t stream);
// whether a product takes the 256 x 256 tile kernel (a non-zero reduction, a multiple of 64)
bool proj_gemm_wide_ok(const ProjGemmParams& p);
// dW = dY^T X (pw) and dX = dY W (px) of the backward in one launch, both on the 256 x 256 tile kernel
hipError_t launch_proj_gemm_bwd_pair(const ProjGemmParams& pw, const ProjGemmParams& px, hipStream_t stream);
hipError_t launch_proj_grad_pack(const void* dq, const void* dk, const void* dv, bool src_f32, bf16* dy,
                                 const int32_t* pos, int64_t rows, int hq, int hkv, bool rotate,
                                 const RopeFreqTable& freq, hipStream_t stream);

}  // namespace ba
