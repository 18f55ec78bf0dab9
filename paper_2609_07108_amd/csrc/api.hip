// C ABI device entry points: validation, upload of the plan tables into the
// caller's workspace, and the launch sequence of one forward / backward call.
#include <mutex>
#include <string>

#include "ba_internal.h"
#include "kernels.h"

namespace ba {
namespace {

int fail(int code, const std::string& msg) {
  set_error(msg);
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(BA_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

hipError_t record(void* ev, hipStream_t stream) {
  return ev ? hipEventRecord(reinterpret_cast<hipEvent_t>(ev), stream) : hipSuccess;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// every device tensor is read in 16-byte vectors
int check_ptr(const void* p, bool needed, const char* name) {
  if (!needed) return BA_OK;
  if (!p) return fail(BA_E_INVAL, std::string(name) + " is NULL");
  if (!aligned16(p)) return fail(BA_E_INVAL, std::string(name) + " is not 16-byte aligned");
  return BA_OK;
}

struct Common {
  int rc = BA_OK;
  WorkspaceLayout w;
  char* ws = nullptr;
};

Common prepare(const ba_plan* plan, int32_t mode, void* workspace, size_t ws_bytes, bool bwd,
               hipStream_t stream) {
  Common c;
  if (!plan) {
    c.rc = fail(BA_E_INVAL, "plan is NULL");
    return c;
  }
  if (mode != BA_MODE_PER_STEP && mode != BA_MODE_FUSED) {
    c.rc = fail(BA_E_INVAL, "unknown mode");
    return c;
  }
  const Plan& P = plan->p;
  if (P.cp_size > kMaxCp) {
    c.rc = fail(BA_E_UNSUPPORTED, "cp_size > 32 unsupported");
    return c;
  }
  c.w = workspace_layout(P, mode);
  const size_t need = bwd ? c.w.bwd_total : c.w.fwd_total;
  if (!workspace || ws_bytes < need) {
    c.rc = fail(BA_E_WORKSPACE, "workspace of " + std::to_string(ws_bytes) + " bytes, need " +
                                    std::to_string(need));
    return c;
  }
  if (((uintptr_t)workspace & 255) != 0) {
    c.rc = fail(BA_E_WORKSPACE, "workspace must be 256-byte aligned");
    return c;
  }
  c.ws = static_cast<char*>(workspace);
  if (!P.image.empty()) {
    hipError_t e = hipMemcpyAsync(c.ws + c.w.tables, P.image.data(), P.image.size(), hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) c.rc = hip_fail(e, "upload of plan tables");
  }
  return c;
}

// Rotary embedding tables of a plan inside the workspace copy of its image.
struct RopeTables {
  const int32_t* pos_block;  // [C][n_local]
  const int32_t* pos_qmain;  // [n_local]
  const int32_t* pos_br;     // [num_branch_rows]
  const RopeFreq* freq;      // turns per position (float pair), gradient rotation
  const double* rad;         // radians per position (double), input rotation
};

RopeTables rope_tables(const Plan& P, const Common& c) {
  const char* t = c.ws + c.w.tables;
  return RopeTables{reinterpret_cast<const int32_t*>(t + P.off_pos_block),
                    reinterpret_cast<const int32_t*>(t + P.off_pos_qmain),
                    reinterpret_cast<const int32_t*>(t + P.off_pos_br),
                    reinterpret_cast<const RopeFreq*>(t + P.off_freq),
                    reinterpret_cast<const double*>(t + P.off_rad)};
}

// Rotated bf16 copies of the queries and keys of one call; the pointers the
// kernels read are redirected to them.
template <typename Params>
hipError_t rotate_inputs(const Plan& P, const Common& c, const void* q_main, const void* q_br, const void* k_br,
                         const void* const* k_step, bool has_main, bool has_br, bool has_keys, Params& p,
                         hipStream_t stream) {
  const RopeTables rt = rope_tables(P, c);
  const int64_t nl = P.n_local, nb = P.num_branch_rows;
  const int64_t krow = (int64_t)P.hkv * kHeadDim;
  hipError_t e = hipSuccess;
  if (has_main) {
    bf16* rq = reinterpret_cast<bf16*>(c.ws + c.w.rq_main);
    if ((e = launch_rope_rows(static_cast<const bf16*>(q_main), rq, rt.pos_qmain, rt.rad, nl, P.hq, stream)))
      return e;
    p.q_main = rq;
  }
  if (has_br) {
    bf16* rq = reinterpret_cast<bf16*>(c.ws + c.w.rq_br);
    bf16* rk = reinterpret_cast<bf16*>(c.ws + c.w.rk_br);
    if ((e = launch_rope_rows(static_cast<const bf16*>(q_br), rq, rt.pos_br, rt.rad, nb, P.hq, stream))) return e;
    if ((e = launch_rope_rows(static_cast<const bf16*>(k_br), rk, rt.pos_br, rt.rad, nb, P.hkv, stream))) return e;
    p.q_br = rq;
    p.k_br = rk;
  }
  for (int j = 0; j < P.cp_size && has_keys; ++j) {
    bf16* rk = reinterpret_cast<bf16*>(c.ws + c.w.rk_step) + (int64_t)j * nl * krow;
    if ((e = launch_rope_rows(static_cast<const bf16*>(k_step[j]), rk, rt.pos_block + (int64_t)j * nl, rt.rad, nl,
                              P.hkv, stream)))
      return e;
    p.k_step[j] = rk;
  }
  return e;
}

}  // namespace
}  // namespace ba

using namespace ba;

extern "C" int branch_attn_fwd(void* stream_, const ba_plan* plan, int32_t mode, const ba_fwd_io* io,
                               void* workspace, size_t workspace_bytes) {
  hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
  if (!io) return fail(BA_E_INVAL, "io is NULL");
  if (!plan) return fail(BA_E_INVAL, "plan is NULL");
  const Plan& P = plan->p;
  mode = resolve_mode(P, mode);
  const bool has_main = P.any_main_query;   // some sequence's main tokens are queries
  const bool has_keys = P.n_local > 0;      // main keys exist
  const bool has_br = P.num_branch_rows > 0 && !P.groups.empty();
  int rc;
  if ((rc = check_ptr(io->q_main, has_main, "q_main")) || (rc = check_ptr(io->o_main, has_main, "o_main")) ||
      (rc = check_ptr(io->lse_main, has_main, "lse_main")) || (rc = check_ptr(io->q_br, has_br, "q_br")) ||
      (rc = check_ptr(io->k_br, has_br, "k_br")) || (rc = check_ptr(io->v_br, has_br, "v_br")) ||
      (rc = check_ptr(io->o_br, has_br, "o_br")) || (rc = check_ptr(io->lse_br, has_br, "lse_br")))
    return rc;
  if (has_keys && (!io->k_step || !io->v_step)) return fail(BA_E_INVAL, "k_step / v_step missing");
  if (P.toks.empty()) return BA_OK;
  Common c = prepare(plan, mode, workspace, workspace_bytes, false, stream);
  if (c.rc) return c.rc;

  FwdParams p{};
  p.seqs = reinterpret_cast<const SeqInfo*>(c.ws + c.w.tables + P.off_seqs);
  p.toks = reinterpret_cast<const TokInfo*>(c.ws + c.w.tables + P.off_toks);
  p.groups = reinterpret_cast<const GroupInfo*>(c.ws + c.w.tables + P.off_groups);
  p.tiles = reinterpret_cast<const FwdTile*>(c.ws + c.w.tables + P.off_fwd);
  p.num_tiles = (int32_t)P.fwd_tiles.size();
  p.br_keys = reinterpret_cast<const int32_t*>(c.ws + c.w.tables + P.off_br_keys);
  p.tok_bslot = reinterpret_cast<const int32_t*>(c.ws + c.w.tables + P.off_bslot);
  p.C = P.cp_size;
  p.rank = P.cp_rank;
  p.hq = P.hq;
  p.hkv = P.hkv;
  p.G = P.group;
  p.num_tokens = (int32_t)P.toks.size();
  p.scale_log2 = P.scale * kLog2e;
  p.n_local = P.n_local;
  p.n_br = P.num_branch_rows;
  p.q_main = static_cast<const bf16*>(io->q_main);
  p.q_br = static_cast<const bf16*>(io->q_br);
  p.k_br = static_cast<const bf16*>(io->k_br);
  p.v_br = static_cast<const bf16*>(io->v_br);
  for (int j = 0; j < P.cp_size && has_keys; ++j) {
    if ((rc = check_ptr(io->k_step[j], has_keys, "k_step[j]")) || (rc = check_ptr(io->v_step[j], has_keys, "v_step[j]")))
      return rc;
    p.k_step[j] = static_cast<const bf16*>(io->k_step[j]);
    p.v_step[j] = static_cast<const bf16*>(io->v_step[j]);
  }
  p.o_main = static_cast<bf16*>(io->o_main);
  p.o_br = static_cast<bf16*>(io->o_br);
  p.lse_main = io->lse_main;
  p.lse_br = io->lse_br;
  hipError_t e;
  if (P.rope_theta > 0.f &&
      (e = rotate_inputs(P, c, io->q_main, io->q_br, io->k_br, io->k_step, has_main, has_br, has_keys, p, stream)))
    return hip_fail(e, "rotary embedding launch");
  if ((e = record(io->ring_begin, stream)) != hipSuccess) return hip_fail(e, "event record");
  if (mode == BA_MODE_FUSED) {
    p.step_first = 0;
    p.step_count = P.cp_size;
    if ((e = launch_fwd(p, kModeFused, stream)) != hipSuccess) return hip_fail(e, "forward launch");
    if ((e = record(io->ring_end, stream)) != hipSuccess) return hip_fail(e, "event record");
    return BA_OK;
  }
  p.o_acc = reinterpret_cast<float*>(c.ws + c.w.o_acc);
  p.lse_acc = reinterpret_cast<float*>(c.ws + c.w.lse_acc);
  for (int i = 0; i < P.cp_size; ++i) {
    p.step_first = i;
    p.step_count = 1;
    p.acc_first = i == 0;
    if ((e = launch_fwd(p, kModeStep, stream)) != hipSuccess) return hip_fail(e, "ring-step launch");
  }
  if ((e = record(io->ring_end, stream)) != hipSuccess) return hip_fail(e, "event record");
  if ((e = launch_fwd_finalize(p, stream)) != hipSuccess) return hip_fail(e, "branch/merge launch");
  return BA_OK;
}

// ------------------------------------------------ forward without allocation
// A file-scope device array stands in for the caller's workspace.  In host
// code its name is only a stand-in for the device object: the address the
// kernels may use is obtained per device with hipGetSymbolAddress, once, with
// that device current, and kept here.
namespace ba {
namespace {
constexpr size_t kNoAllocScratchBytes = size_t(64) << 20;
constexpr int kMaxDevices = 64;
}  // namespace
}  // namespace ba

static __device__ __align__(256) char scratch[ba::kNoAllocScratchBytes];

namespace ba {
namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// address of this device's copy of `scratch` (looked up on first use)
int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(BA_E_UNSUPPORTED, "device index beyond 63");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!ptr || ((uintptr_t)ptr & 255) != 0) return fail(BA_E_HIP, "scratch address is NULL or misaligned");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return BA_OK;
}
}  // namespace
}  // namespace ba

extern "C" int branch_attn_fwd_noalloc(void* stream, const ba_plan* plan, int32_t mode, const ba_fwd_io* io) {
  if (!plan) return fail(BA_E_INVAL, "plan is NULL");
  if (mode != BA_MODE_PER_STEP && mode != BA_MODE_FUSED && mode != BA_MODE_AUTO)
    return fail(BA_E_INVAL, "unknown mode");
  const Plan& P = plan->p;
  mode = resolve_mode(P, mode);
  if (P.cp_size > kMaxCp) return fail(BA_E_UNSUPPORTED, "cp_size > 32 unsupported");
  const size_t need = workspace_layout(P, mode).fwd_total;
  if (need > kNoAllocScratchBytes)
    return fail(BA_E_WORKSPACE, "branch_attn_fwd_noalloc: this plan and mode need " + std::to_string(need) +
                                    " bytes of scratch, the static scratch holds " +
                                    std::to_string(kNoAllocScratchBytes) +
                                    " (use BA_MODE_FUSED without rotary embedding, or branch_attn_fwd)");
  void* ws = nullptr;
  int rc = scratch_address(&ws);
  if (rc) return rc;
  return branch_attn_fwd(stream, plan, mode, io, ws, kNoAllocScratchBytes);
}

extern "C" int branch_attn_bwd(void* stream_, const ba_plan* plan, int32_t mode, const ba_bwd_io* io,
                               void* workspace, size_t workspace_bytes) {
  hipStream_t stream = reinterpret_cast<hipStream_t>(stream_);
  if (!io) return fail(BA_E_INVAL, "io is NULL");
  if (!plan) return fail(BA_E_INVAL, "plan is NULL");
  const Plan& P = plan->p;
  mode = resolve_mode(P, mode);
  const bool has_main = P.any_main_query;
  const bool has_keys = P.n_local > 0;
  const bool has_br = P.num_branch_rows > 0 && !P.groups.empty();
  if (io->grad_dtype != BA_DTYPE_BF16 && io->grad_dtype != BA_DTYPE_F32)
    return fail(BA_E_INVAL, "grad_dtype must be BA_DTYPE_BF16 or BA_DTYPE_F32");
  int rc;
  if ((rc = check_ptr(io->q_main, has_main, "q_main")) || (rc = check_ptr(io->o_main, has_main, "o_main")) ||
      (rc = check_ptr(io->lse_main, has_main, "lse_main")) || (rc = check_ptr(io->do_main, has_main, "do_main")) ||
      (rc = check_ptr(io->dq_main, has_main, "dq_main")) || (rc = check_ptr(io->q_br, has_br, "q_br")) ||
      (rc = check_ptr(io->k_br, has_br, "k_br")) || (rc = check_ptr(io->v_br, has_br, "v_br")) ||
      (rc = check_ptr(io->o_br, has_br, "o_br")) || (rc = check_ptr(io->lse_br, has_br, "lse_br")) ||
      (rc = check_ptr(io->do_br, has_br, "do_br")) || (rc = check_ptr(io->dq_br, has_br, "dq_br")) ||
      (rc = check_ptr(io->dk_br, has_br, "dk_br")) || (rc = check_ptr(io->dv_br, has_br, "dv_br")))
    return rc;
  if (has_keys && (!io->k_step || !io->v_step || !io->dk_step || !io->dv_step))
    return fail(BA_E_INVAL, "k_step / v_step / dk_step / dv_step missing");
  Common c{};
  if (P.cp_size > kMaxCp) return fail(BA_E_UNSUPPORTED, "cp_size > 32 unsupported");
  BwdParams p{};
  hipError_t e;
  // the per-step KV gradients are overwritten: clear the rows no work item writes
  const size_t elem = io->grad_dtype == BA_DTYPE_F32 ? 4 : 2;
  const size_t step_bytes = (size_t)P.n_local * P.hkv * kHeadDim * elem;
  for (int j = 0; j < P.cp_size && has_keys; ++j) {
    if ((rc = check_ptr(io->k_step[j], true, "k_step[j]")) || (rc = check_ptr(io->v_step[j], true, "v_step[j]")) ||
        (rc = check_ptr(io->dk_step[j], true, "dk_step[j]")) || (rc = check_ptr(io->dv_step[j], true, "dv_step[j]")))
      return rc;
    p.k_step[j] = static_cast<const bf16*>(io->k_step[j]);
    p.v_step[j] = static_cast<const bf16*>(io->v_step[j]);
    p.dk_step[j] = io->dk_step[j];
    p.dv_step[j] = io->dv_step[j];
  }
  if (P.toks.empty() && !has_keys) return BA_OK;
  c = prepare(plan, mode, workspace, workspace_bytes, true, stream);
  if (c.rc) return c.rc;
  const bool rope = P.rope_theta > 0.f;
  const int64_t krow = (int64_t)P.hkv * kHeadDim;
  float* gk_step = rope ? reinterpret_cast<float*>(c.ws + c.w.gk_step) : nullptr;
  float* gv_step = rope ? reinterpret_cast<float*>(c.ws + c.w.gv_step) : nullptr;
  for (int j = 0; j < P.cp_size && has_keys; ++j) {
    if (rope && !P.toks.empty()) {
      // gradients of the rotated keys are staged in fp32 and rotated back at the end
      p.dk_step[j] = gk_step + (int64_t)j * P.n_local * krow;
      p.dv_step[j] = gv_step + (int64_t)j * P.n_local * krow;
      const size_t f32_bytes = (size_t)P.n_local * krow * sizeof(float);
      if ((e = launch_zero(p.dk_step[j], f32_bytes, stream)) != hipSuccess) return hip_fail(e, "clear dk");
      if ((e = launch_zero(p.dv_step[j], f32_bytes, stream)) != hipSuccess) return hip_fail(e, "clear dv");
    } else {
      if ((e = launch_zero(io->dk_step[j], step_bytes, stream)) != hipSuccess) return hip_fail(e, "clear dk");
      if ((e = launch_zero(io->dv_step[j], step_bytes, stream)) != hipSuccess) return hip_fail(e, "clear dv");
    }
  }
  if (P.toks.empty()) return BA_OK;
  p.seqs = reinterpret_cast<const SeqInfo*>(c.ws + c.w.tables + P.off_seqs);
  p.toks = reinterpret_cast<const TokInfo*>(c.ws + c.w.tables + P.off_toks);
  p.groups = reinterpret_cast<const GroupInfo*>(c.ws + c.w.tables + P.off_groups);
  const BwdTile* tiles = reinterpret_cast<const BwdTile*>(c.ws + c.w.tables + P.off_bwd);
  p.qtiles = reinterpret_cast<const FwdTile*>(c.ws + c.w.tables + P.off_fwd);
  p.num_qtiles = (int32_t)P.fwd_tiles.size();
  p.br_keys = reinterpret_cast<const int32_t*>(c.ws + c.w.tables + P.off_br_keys);
  p.tok_bslot = reinterpret_cast<const int32_t*>(c.ws + c.w.tables + P.off_bslot);
  p.C = P.cp_size;
  p.rank = P.cp_rank;
  p.hq = P.hq;
  p.hkv = P.hkv;
  p.G = P.group;
  p.num_tokens = (int32_t)P.toks.size();
  p.num_groups = (int32_t)P.groups.size();
  p.scale = P.scale;
  p.scale_log2 = P.scale * kLog2e;
  p.n_local = P.n_local;
  p.n_br = P.num_branch_rows;
  p.q_main = static_cast<const bf16*>(io->q_main);
  p.q_br = static_cast<const bf16*>(io->q_br);
  p.k_br = static_cast<const bf16*>(io->k_br);
  p.v_br = static_cast<const bf16*>(io->v_br);
  p.o_main = static_cast<const bf16*>(io->o_main);
  p.o_br = static_cast<const bf16*>(io->o_br);
  p.lse_main = io->lse_main;
  p.lse_br = io->lse_br;
  p.do_main = static_cast<const bf16*>(io->do_main);
  p.do_br = static_cast<const bf16*>(io->do_br);
  p.dq_main = io->dq_main;
  p.dq_br = io->dq_br;
  p.dk_br = io->dk_br;
  p.dv_br = io->dv_br;
  p.grad_f32 = io->grad_dtype == BA_DTYPE_F32;
  p.rowstat = reinterpret_cast<float2*>(c.ws + c.w.rowstat);
  p.qtok = reinterpret_cast<bf16*>(c.ws + c.w.qtok);
  p.gtok = reinterpret_cast<bf16*>(c.ws + c.w.gtok);
  p.dq_acc = mode == BA_MODE_PER_STEP ? reinterpret_cast<float*>(c.ws + c.w.dq_acc) : nullptr;
  p.kv_part = P.kv_slots > 0 ? reinterpret_cast<float*>(c.ws + c.w.kv_part) : nullptr;
  p.splits = reinterpret_cast<const KvSplit*>(c.ws + c.w.tables + P.off_splits);
  p.num_splits = (int32_t)P.kv_splits.size();
  if (rope) {
    if ((e = rotate_inputs(P, c, io->q_main, io->q_br, io->k_br, io->k_step, has_main, has_br, has_keys, p, stream)))
      return hip_fail(e, "rotary embedding launch");
    p.dq_main = c.ws + c.w.gq_main;
    p.dq_br = c.ws + c.w.gq_br;
    p.dk_br = c.ws + c.w.gk_br;
    p.dv_br = c.ws + c.w.gv_br;
    p.grad_f32 = 1;
  }

  if ((e = launch_bwd_preprocess(p, stream)) != hipSuccess) return hip_fail(e, "preprocess launch");
  if ((e = record(io->ring_begin, stream)) != hipSuccess) return hip_fail(e, "event record");
  // ring replay of dK/dV: one launch per ring step, the arriving block's
  // work items (returned to its owner in a real ring), in both schedules:
  // a launch's items then start together and walk their query tiles in step
  // (see the planner's walk directions), which one launch over every step's
  // items does not keep (measured 1-3 % slower)
  for (int i = 0; i < P.cp_size; ++i) {
    p.tiles = tiles + P.bwd_step_off[i];
    p.num_tiles = P.bwd_step_off[i + 1] - P.bwd_step_off[i];
    if ((e = launch_bwd_kv(p, stream)) != hipSuccess) return hip_fail(e, "ring-step dK/dV launch");
  }
  if ((e = launch_bwd_kv_reduce(p, stream)) != hipSuccess) return hip_fail(e, "dK/dV partial-sum launch");
  if ((e = record(io->kv_end, stream)) != hipSuccess) return hip_fail(e, "event record");
  if (mode == BA_MODE_FUSED) {
    // dQ over every step in one pass
    p.step_first = 0;
    p.step_count = P.cp_size;
    if ((e = launch_bwd_dq(p, kModeFused, stream)) != hipSuccess) return hip_fail(e, "dQ launch");
    if ((e = record(io->ring_end, stream)) != hipSuccess) return hip_fail(e, "event record");
  } else {
    // per ring step this rank's dQ sums
    for (int i = 0; i < P.cp_size; ++i) {
      p.step_first = i;
      p.step_count = 1;
      p.acc_first = i == 0;
      if ((e = launch_bwd_dq(p, kModeStep, stream)) != hipSuccess) return hip_fail(e, "ring-step dQ launch");
    }
    if ((e = record(io->ring_end, stream)) != hipSuccess) return hip_fail(e, "event record");
    if ((e = launch_bwd_dq_finalize(p, stream)) != hipSuccess) return hip_fail(e, "dQ finalize launch");
  }
  if (has_br) {
    if ((e = launch_bwd_branch(p, P.max_group_len, stream)) != hipSuccess) return hip_fail(e, "branch backward launch");
  }
  if (rope) {
    // gradients with respect to the unrotated queries and keys: the
    // transposed rotation of the staged ones (values were not rotated)
    const RopeTables rt = rope_tables(P, c);
    const bool f32 = io->grad_dtype == BA_DTYPE_F32;
    const int64_t nl = P.n_local, nb = P.num_branch_rows;
    auto grad = [&](const void* src, void* dst, const int32_t* pos, int64_t rows, int heads, bool rot) {
      return launch_rope_grad(static_cast<const float*>(src), dst, f32, pos, rt.freq, rows, heads, rot, stream);
    };
    if (has_main && (e = grad(p.dq_main, io->dq_main, rt.pos_qmain, nl, P.hq, true)))
      return hip_fail(e, "rotary gradient launch");
    if (has_br && ((e = grad(p.dq_br, io->dq_br, rt.pos_br, nb, P.hq, true)) ||
                   (e = grad(p.dk_br, io->dk_br, rt.pos_br, nb, P.hkv, true)) ||
                   (e = grad(p.dv_br, io->dv_br, rt.pos_br, nb, P.hkv, false))))
      return hip_fail(e, "rotary gradient launch");
    for (int j = 0; j < P.cp_size && has_keys; ++j)
      if ((e = grad(p.dk_step[j], io->dk_step[j], rt.pos_block + j * nl, nl, P.hkv, true)) ||
          (e = grad(p.dv_step[j], io->dv_step[j], rt.pos_block + j * nl, nl, P.hkv, false)))
        return hip_fail(e, "rotary gradient launch");
  }
  return BA_OK;
}
