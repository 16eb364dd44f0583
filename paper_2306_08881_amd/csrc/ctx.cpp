// C ABI of the ACP-SGD compressor: context, state binding, step sequencing and launches.
// Every argument, state and sequencing check runs on the host before anything is enqueued.
#include <hip/hip_runtime.h>

#include <cstring>
#include <string>
#include <vector>

#include "acp.h"
#include "plan.hpp"

namespace acp {
hipError_t launch(const Launch& l, int32_t rank, const KArgs& args, hipStream_t s);
// address of the static Q-step scratch on `device`, which must be the current device
hipError_t scratch_address(int device, float** out);
}

struct acp_ctx {
  acp::Plan plan;
  uint64_t seed = 0;
  int32_t world = 1;
  uint32_t flags = 0;
  int32_t num_tensors = 0;
  std::vector<float> init_fac;  // host image of the factor region holding P_0 and Q_0

  uint8_t* dev = nullptr;       // bound state block
  int64_t dev_bytes = 0;
  int device = -1;
  float* scratch = nullptr;     // the bound device's static Q-step scratch (acp_compress_noalloc)
  std::string scratch_err;      // why it is null after a bind
  // a second stream (default priority) and fork / join events on the bound device: the rank-4
  // P-step's class launches after the first run there, beside it
  hipStream_t side = nullptr;
  hipEvent_t fork_ev = nullptr, join_ev = nullptr;
  std::vector<int64_t> last_step;   // per bucket: last completed step
  std::vector<int64_t> pending;     // per bucket: compressed step awaiting decompress (0 = none)
  std::vector<uint8_t> deferred;    // per bucket: E form of the arena (kExplicit, kHoldsF, kHoldsX)
  std::vector<uint8_t> phase;       // per bucket, Power-SGD: 1 after the first half, 2 after the second
  // per bucket: the step whose compress finds its orthogonal factor (K_APPLY's Qh or Ph) already
  // formed, beside the previous decompress (0: none)
  std::vector<int64_t> applied;
  mutable std::string err;

  // kernel timing (acp_profile_start / acp_profile_stop)
  int32_t prof_family = 0;
  std::vector<hipEvent_t> prof_events;  // begin, end pairs
  int64_t prof_used = 0;
  double prof_bytes = 0.0;
};

namespace {

constexpr uint64_t kMagic = 0x3153504341ull;  // "ACPS1"
constexpr int64_t kVersion = 1;

// What the E arena of a bucket holds: E itself, F = M' after a Q-step (E = F - Ph Ql^T), or
// X = M' after a P-step of rank >= 8 (E = X - Pl Qh^T).
constexpr uint8_t kExplicit = 0, kHoldsF = 1, kHoldsX = 2;

uint8_t form_after_compress(const acp_ctx* c, int64_t step) {
  if (!c->plan.ef) return kExplicit;
  if (!(step & 1)) return kHoldsF;
  return c->plan.rank >= acp::kWideRank ? kHoldsX : kExplicit;
}

// the masks of KArgs for bucket slot i (bucket base + i)
void set_form(acp::KArgs& a, int32_t i, uint8_t form) {
  if (form == kHoldsF) a.deferred |= 1ull << i;
  if (form == kHoldsX) a.deferred_p |= 1ull << i;
}

acp_status fail(const acp_ctx* c, acp_status s, const std::string& msg) {
  if (c) c->err = msg;
  return s;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

acp_status check_device(const acp_ctx* c) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(c, ACP_E_DEVICE, "hipGetDevice failed");
  if (dev != c->device)
    return fail(c, ACP_E_INVALID, "the device current at bind time must be current for this call");
  return ACP_OK;
}

acp::KArgs base_args(const acp_ctx* c) {
  const acp::Plan& p = c->plan;
  acp::KArgs a{};
  uint8_t* d = c->dev;
  a.e = reinterpret_cast<float*>(d + p.off_e);
  a.fac = reinterpret_cast<float*>(d + p.off_fac);
  a.w = reinterpret_cast<double*>(d + p.off_w);
  a.gpart = reinterpret_cast<double*>(d + p.off_gpart);
  a.qpart = reinterpret_cast<float*>(d + p.off_qpart);
  a.mats = reinterpret_cast<const acp::MatDesc*>(d + p.off_mats);
  a.vecs = reinterpret_cast<const acp::VecDesc*>(d + p.off_vecs);
  a.ef = p.ef ? 1 : 0;
  a.inv_p = 1.0f / static_cast<float>(c->world);
  a.seed = c->seed;
  return a;
}

bool overlaps(const void* x, int64_t x_floats, const void* y, int64_t y_floats) {
  const char* a = static_cast<const char*>(x);
  const char* b = static_cast<const char*>(y);
  return a < b + y_floats * 4 && b < a + x_floats * 4;
}

// A run of two or more consecutive rank-4 P-step launches (K_PFUSED: one per column class, on
// disjoint matrices, none reading what another writes) from launch i on, each moving less than
// kOverlapBytes: their tails are a large part of their time, which running them side by side
// fills (larger launches slowed each other down when run so: BERT-base and BERT-large).
constexpr double kOverlapBytes = 512.0 * (1 << 20);
bool small_pstep_run(const std::vector<acp::Launch>& launches, size_t i) {
  size_t k = i;
  while (k < launches.size() && launches[k].kernel == acp::K_PFUSED) {
    if (launches[k].alg_bytes >= kOverlapBytes) return false;
    ++k;
  }
  return k - i >= 2;
}

// The Gram finish of the aggregated factor (K_WFACT, then K_GSUM and K_CHOL) after a rank 8-256
// decompress launch (K_WRECON): it reads the aggregated factor only and writes the factor slot,
// the Gram partials, W and the raw vectors' part of the output, none of which the decompress
// reads or writes, so it runs on the side stream beside the decompress (its few workgroups and
// dependent launches are latency-bound, the decompress is bound by HBM writes).  From
// kBlockedRank on the Gram's matrix-core work slowed the decompress beside it by more than the
// overlap saved (BERT-large r=128), so those ranks keep the one stream.
bool orth_kernel(int32_t k) { return k == acp::K_WFACT || k == acp::K_GSUM || k == acp::K_CHOL; }
bool orth_after_recon(const acp_ctx* c, const std::vector<acp::Launch>& launches, size_t i) {
  return c->plan.rank < acp::kBlockedRank && launches[i].kernel == acp::K_WRECON &&
         i + 1 < launches.size() && launches[i + 1].kernel == acp::K_WFACT;
}

// Enqueues `launches` on s; skip_chol leaves out the Gram finish (K_GSUM, K_CHOL), which factor
// tiles that only copy (KArgs::copy_only) do not need, and skip_apply the orthogonal factor's
// product (K_APPLY), when the previous decompress formed it.  Two kinds of run are split over two
// streams, their first launch on s and the others on the context's side stream, forked from s
// before the run and joined back into s after it (the joins keep graph capture on s whole): a
// small P-step run (small_pstep_run) and a decompress with the Gram finish after it
// (orth_after_recon).  In the latter, `apply` (the next compress's K_APPLY, or null) follows the
// Gram finish on the side stream, and *applied tells whether it was enqueued.
struct RunOpts {
  bool skip_chol = false;
  bool skip_apply = false;
  const acp::Launch* apply = nullptr;
  bool* applied = nullptr;
};
acp_status run(const acp_ctx* c, const std::vector<acp::Launch>& launches, acp::KArgs a,
               hipStream_t s, const RunOpts& o = RunOpts{}) {
  const acp::Tile* tiles = reinterpret_cast<const acp::Tile*>(c->dev + c->plan.off_tiles);
  acp_ctx* mc = const_cast<acp_ctx*>(c);
  const hipStream_t s0 = s;
  enum { kNone, kPstep, kOrth } forked = kNone;  // the run whose later launches go to the side
  if (o.applied) *o.applied = false;
  // one launch of the list (or o.apply) on stream st
  auto enqueue = [&](const acp::Launch& l, hipStream_t st) -> std::string {
    a.tiles = tiles + l.tile_off;
    a.ntiles = l.ntiles;
    a.variant = l.variant;
    const bool timed = mc->prof_family != 0 && l.family == mc->prof_family &&
                       2 * mc->prof_used < static_cast<int64_t>(mc->prof_events.size());
    if (timed && hipEventRecord(mc->prof_events[2 * mc->prof_used], st) != hipSuccess)
      return "hipEventRecord failed";
    const hipError_t e = acp::launch(l, c->plan.rank, a, st);
    if (e != hipSuccess) return std::string("kernel launch failed: ") + hipGetErrorString(e);
    if (timed) {
      if (hipEventRecord(mc->prof_events[2 * mc->prof_used + 1], st) != hipSuccess)
        return "hipEventRecord failed";
      mc->prof_used += 1;
      mc->prof_bytes += l.alg_bytes;
    }
    return "";
  };
  // the Gram finish's run ends with o.apply on the side stream; then s0 waits for the side
  // stream's work (also before an error return)
  std::string apply_err;
  auto join = [&](bool with_apply = true) -> bool {
    if (with_apply && forked == kOrth && o.apply && apply_err.empty()) {
      apply_err = enqueue(*o.apply, c->side);
      if (apply_err.empty() && o.applied) *o.applied = true;
    }
    forked = kNone;
    s = s0;
    const bool ok = hipEventRecord(c->join_ev, c->side) == hipSuccess && hipStreamWaitEvent(s0, c->join_ev, 0) == hipSuccess;
    return ok && apply_err.empty();
  };
  auto error = [&](const std::string& msg) {
    if (forked != kNone) (void)join(false);
    return fail(c, ACP_E_DEVICE, msg);
  };
  for (size_t i = 0; i < launches.size(); ++i) {
    const acp::Launch& l = launches[i];
    if (o.skip_chol && (l.kernel == acp::K_GSUM || l.kernel == acp::K_CHOL)) continue;
    if (o.skip_apply && l.kernel == acp::K_APPLY) continue;
    const bool pstep = l.kernel == acp::K_PFUSED;
    const bool continues = (forked == kPstep && pstep) || (forked == kOrth && orth_kernel(l.kernel));
    if (forked != kNone && !continues && !join())
      return fail(c, ACP_E_DEVICE, apply_err.empty() ? "side stream join failed" : apply_err);
    const bool fork_p = forked == kNone && pstep && c->side && small_pstep_run(launches, i);
    const bool fork_o = forked == kNone && !fork_p && c->side && orth_after_recon(c, launches, i);
    if (fork_p || fork_o) {
      if (hipEventRecord(c->fork_ev, s0) != hipSuccess || hipStreamWaitEvent(c->side, c->fork_ev, 0) != hipSuccess)
        return fail(c, ACP_E_DEVICE, "side stream fork failed");  // nothing is on the side yet
      forked = fork_p ? kPstep : kOrth;
      s = s0;  // this first launch of the run stays on s, the rest go to the side
    } else if (forked != kNone) {
      s = c->side;
    }
    const std::string msg = enqueue(l, s);
    if (!msg.empty()) return error(msg);
  }
  if (forked != kNone && !join())
    return fail(c, ACP_E_DEVICE, apply_err.empty() ? "side stream join failed" : apply_err);
  return ACP_OK;
}

void release_side(acp_ctx* c) {
  if (c->side) (void)hipStreamDestroy(c->side);
  if (c->fork_ev) (void)hipEventDestroy(c->fork_ev);
  if (c->join_ev) (void)hipEventDestroy(c->join_ev);
  c->side = nullptr;
  c->fork_ev = c->join_ev = nullptr;
}

int64_t checkpoint_payload(const acp::Plan& p) {
  return p.e_floats * 4 + p.fac_floats * 4 + p.w_doubles * 8;
}

struct CkptHeader {
  uint64_t magic;
  int64_t version;
  int64_t num_tensors, rank, cap, world, flags, nbuckets, seed;
  int64_t e_floats, fac_floats, w_doubles;
};

// The K_APPLY launch that opens a compress list (the orthogonal factor Qh = Q W or Ph = P W of
// the reused factor), when the previous decompress may form it beside its own launches instead:
// reused factors only (with fresh draws the factor is drawn in the compress call).
const acp::Launch* leading_apply(const acp_ctx* c, const std::vector<acp::Launch>& compress) {
  if (!c->plan.reuse || c->plan.psgd || compress.empty() || compress[0].kernel != acp::K_APPLY) return nullptr;
  return &compress[0];
}

// acp_compress and acp_compress_noalloc: checks, then the bucket's compress launches.  `qpart`,
// when not null, replaces the state block's Q-step partial region as the kernels' base.
acp_status compress_bucket(acp_ctx* c, int64_t step, int32_t b, const float* grad, float* factor_buf,
                           void* stream, float* qpart) {
  if (!c) return ACP_E_INVALID;
  if (c->plan.psgd) return fail(c, ACP_E_UNSUPPORTED, "this context runs Power-SGD (acp_powersgd_*)");
  if (!c->dev) return fail(c, ACP_E_STATE, "state not bound");
  if (b < 0 || b >= static_cast<int32_t>(c->plan.buckets.size()))
    return fail(c, ACP_E_INVALID, "bucket index out of range");
  if (!grad || !factor_buf) return fail(c, ACP_E_INVALID, "null buffer");
  if (!aligned16(grad) || !aligned16(factor_buf)) return fail(c, ACP_E_INVALID, "buffers must be 16-byte aligned");
  if (c->pending[b] != 0)
    return fail(c, ACP_E_STEP, "compress called twice without decompress");
  if (step != c->last_step[b] + 1)
    return fail(c, ACP_E_STEP, "step " + std::to_string(step) + " out of order (expected " +
                                   std::to_string(c->last_step[b] + 1) + ")");
  const acp::BucketPlan& bk = c->plan.buckets[b];
  {
    const char* g0 = reinterpret_cast<const char*>(grad);
    const char* f0 = reinterpret_cast<const char*>(factor_buf);
    const int64_t fe = (step & 1) ? bk.fac_elems_p : bk.fac_elems_q;
    if (g0 < f0 + fe * 4 && f0 < g0 + bk.grad_elems * 4)
      return fail(c, ACP_E_INVALID, "factor_buf overlaps grad");
  }
  const acp_status ds = check_device(c);
  if (ds != ACP_OK) return ds;
  acp::KArgs a = base_args(c);
  if (qpart) a.qpart = qpart;
  a.base = b;
  a.src[0] = grad;
  a.dst[0] = factor_buf;
  a.parity = static_cast<int32_t>(step & 1);
  a.step = step;
  set_form(a, 0, c->deferred[b]);
  if (!c->plan.reuse) {
    const acp_status sd = run(c, bk.draw[step & 1], a, static_cast<hipStream_t>(stream));
    if (sd != ACP_OK) return sd;
  }
  RunOpts o;
  o.skip_apply = c->applied[b] == step;
  const acp_status st = run(c, bk.compress[step & 1], a, static_cast<hipStream_t>(stream), o);
  if (st != ACP_OK) return st;
  c->pending[b] = step;
  c->deferred[b] = form_after_compress(c, step);
  c->applied[b] = 0;
  return ACP_OK;
}

// Power-SGD: the bucket's image of M' in the E arena (the source of both products with error
// feedback), else the gradient itself
const float* psgd_source(const acp_ctx* c, int32_t b, const float* grad) {
  if (!c->plan.ef) return grad;
  return reinterpret_cast<const float*>(c->dev + c->plan.off_e) + c->plan.buckets[b].e_base;
}

// checks shared by the Power-SGD calls: context, bucket, phase of the step
acp_status psgd_ready(const acp_ctx* c, int64_t step, int32_t b, int32_t phase) {
  if (!c->plan.psgd) return fail(c, ACP_E_UNSUPPORTED, "this context runs ACP-SGD (acp_compress)");
  if (!c->dev) return fail(c, ACP_E_STATE, "state not bound");
  if (b < 0 || b >= static_cast<int32_t>(c->plan.buckets.size()))
    return fail(c, ACP_E_INVALID, "bucket index out of range");
  const bool ok = phase == 0 ? (c->pending[b] == 0 && step == c->last_step[b] + 1)
                             : (c->pending[b] == step && c->phase[b] == phase);
  if (!ok) {
    static const char* what[3] = {"acp_powersgd_p", "acp_powersgd_q", "acp_powersgd_decompress"};
    return fail(c, ACP_E_STEP, std::string(what[phase]) + "(" + std::to_string(step) + ") on bucket " +
                                   std::to_string(b) + " out of order");
  }
  return ACP_OK;
}

acp_status psgd_p_bucket(acp_ctx* c, int64_t step, int32_t b, const float* grad, float* p_buf, hipStream_t s) {
  const acp::BucketPlan& bk = c->plan.buckets[b];
  acp::KArgs a = base_args(c);
  a.base = b;
  a.src[0] = grad;
  a.parity = 1;
  set_form(a, 0, c->deferred[b]);
  acp_status st = run(c, bk.psgd_image, a, s);
  if (st != ACP_OK) return st;
  acp::KArgs m = base_args(c);
  m.ef = 0;
  m.base = b;
  m.src[0] = psgd_source(c, b, grad);
  m.dst[0] = p_buf;
  m.parity = 1;
  return run(c, bk.compress[1], m, s);
}

acp_status psgd_q_bucket(acp_ctx* c, int32_t b, const float* grad, const float* p_agg, float* q_buf,
                         hipStream_t s) {
  const acp::BucketPlan& bk = c->plan.buckets[b];
  acp::KArgs a = base_args(c);
  a.base = b;
  a.src[0] = p_agg;
  a.parity = 0;
  acp_status st = run(c, bk.psgd_fact, a, s);
  if (st != ACP_OK) return st;
  acp::KArgs m = base_args(c);
  m.ef = 0;
  m.base = b;
  m.src[0] = psgd_source(c, b, grad);
  m.dst[0] = q_buf;
  m.parity = 0;
  return run(c, bk.compress[0], m, s);
}

}  // namespace

extern "C" {

acp_status acp_init(acp_ctx** out, int32_t num_tensors, const int32_t* ndims, const int64_t* dims,
                    int32_t rank, uint64_t seed, int64_t bucket_cap_bytes, int32_t world_size,
                    uint32_t flags) {
  if (!out) return ACP_E_INVALID;
  *out = nullptr;
  if (world_size < 1) return ACP_E_INVALID;
  if (flags & ~(ACP_FLAG_EF | ACP_FLAG_REUSE | ACP_FLAG_POWERSGD)) return ACP_E_INVALID;
  const bool reuse = (flags & ACP_FLAG_REUSE) != 0, psgd = (flags & ACP_FLAG_POWERSGD) != 0;
  if (psgd && !reuse) return ACP_E_UNSUPPORTED;
  acp_ctx* c = new acp_ctx();
  const std::string msg = acp::build_plan(c->plan, num_tensors, ndims, dims, rank, bucket_cap_bytes,
                                          (flags & ACP_FLAG_EF) != 0, reuse, psgd);
  if (!msg.empty()) {
    delete c;
    return ACP_E_INVALID;
  }
  c->seed = seed;
  c->world = world_size;
  c->flags = flags;
  c->num_tensors = num_tensors;
  c->init_fac.assign(static_cast<size_t>(c->plan.fac_floats), 0.0f);
  for (int32_t tid = 0; tid < num_tensors; ++tid) {
    const acp::TensorPlan& t = c->plan.tensors[tid];
    if (t.mat < 0) continue;
    const acp::MatDesc& d = c->plan.mats[t.mat];
    acp::draw_init_factor(seed, tid, 0, t.n * rank, c->init_fac.data() + d.p_slot);
    acp::draw_init_factor(seed, tid, 1, t.m * rank, c->init_fac.data() + d.q_slot);
  }
  const size_t nb = c->plan.buckets.size();
  c->last_step.assign(nb, 0);
  c->pending.assign(nb, 0);
  c->deferred.assign(nb, 0);
  c->phase.assign(nb, 0);
  c->applied.assign(nb, 0);
  *out = c;
  return ACP_OK;
}

acp_status acp_state_bytes(const acp_ctx* c, int64_t* bytes) {
  if (!c || !bytes) return fail(c, ACP_E_INVALID, "null argument");
  *bytes = c->plan.total_bytes;
  return ACP_OK;
}

acp_status acp_bind_state(acp_ctx* c, void* device_ptr, int64_t bytes, void* stream) {
  if (!c) return ACP_E_INVALID;
  if (!device_ptr) return fail(c, ACP_E_INVALID, "device_ptr is NULL");
  if ((reinterpret_cast<uintptr_t>(device_ptr) & 255u) != 0)
    return fail(c, ACP_E_INVALID, "state block must be 256-byte aligned");
  if (bytes < c->plan.total_bytes) return fail(c, ACP_E_STATE, "state block too small");
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(c, ACP_E_DEVICE, "hipGetDevice failed");
  const acp::Plan& p = c->plan;
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* d = static_cast<uint8_t*>(device_ptr);
  hipError_t e = hipSuccess;
  if (p.e_floats) e = hipMemsetAsync(d + p.off_e, 0, p.e_floats * 4, s);
  if (e == hipSuccess && p.fac_floats)
    e = hipMemcpyAsync(d + p.off_fac, c->init_fac.data(), p.fac_floats * 4, hipMemcpyHostToDevice, s);
  if (e == hipSuccess && !p.mats.empty())
    e = hipMemcpyAsync(d + p.off_mats, p.mats.data(), p.mats.size() * sizeof(acp::MatDesc),
                       hipMemcpyHostToDevice, s);
  if (e == hipSuccess && !p.vecs.empty())
    e = hipMemcpyAsync(d + p.off_vecs, p.vecs.data(), p.vecs.size() * sizeof(acp::VecDesc),
                       hipMemcpyHostToDevice, s);
  if (e == hipSuccess && !p.tiles.empty())
    e = hipMemcpyAsync(d + p.off_tiles, p.tiles.data(), p.tiles.size() * sizeof(acp::Tile),
                       hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return fail(c, ACP_E_DEVICE, std::string("upload failed: ") + hipGetErrorString(e));
  c->dev = d;
  c->dev_bytes = bytes;
  c->device = dev;
  c->applied.assign(p.buckets.size(), 0);
  acp::KArgs a = base_args(c);
  const acp_status st = run(c, p.gram_init, a, s);
  if (st != ACP_OK) {
    c->dev = nullptr;
    return st;
  }
  e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    c->dev = nullptr;
    return fail(c, ACP_E_DEVICE, std::string("bind failed: ") + hipGetErrorString(e));
  }
  std::fill(c->last_step.begin(), c->last_step.end(), 0);
  std::fill(c->pending.begin(), c->pending.end(), 0);
  std::fill(c->deferred.begin(), c->deferred.end(), 0);
  std::fill(c->phase.begin(), c->phase.end(), 0);
  // the side stream, on the bound device
  release_side(c);
  if (hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&c->fork_ev, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->join_ev, hipEventDisableTiming) != hipSuccess) {
    release_side(c);
    c->dev = nullptr;
    return fail(c, ACP_E_DEVICE, "side stream creation failed");
  }
  // the static scratch of acp_compress_noalloc: looked up once per device, with it current
  c->scratch = nullptr;
  c->scratch_err.clear();
  e = acp::scratch_address(dev, &c->scratch);
  if (e != hipSuccess) {
    c->scratch = nullptr;
    c->scratch_err = std::string("hipGetSymbolAddress of the static scratch failed: ") + hipGetErrorString(e);
  }
  c->err.clear();
  return ACP_OK;
}

int32_t acp_num_buckets(const acp_ctx* c) {
  return c ? static_cast<int32_t>(c->plan.buckets.size()) : -1;
}

acp_status acp_bucket_info(const acp_ctx* c, int32_t b, int32_t* num_tensors, int64_t* grad_elems,
                           int64_t* factor_elems_p, int64_t* factor_elems_q) {
  if (!c) return ACP_E_INVALID;
  if (b < 0 || b >= static_cast<int32_t>(c->plan.buckets.size()))
    return fail(c, ACP_E_INVALID, "bucket index out of range");
  const acp::BucketPlan& bk = c->plan.buckets[b];
  if (num_tensors) *num_tensors = static_cast<int32_t>(bk.tids.size());
  if (grad_elems) *grad_elems = bk.grad_elems;
  if (factor_elems_p) *factor_elems_p = bk.fac_elems_p;
  if (factor_elems_q) *factor_elems_q = bk.fac_elems_q;
  return ACP_OK;
}

acp_status acp_layout(const acp_ctx* c, int32_t b, int32_t* tensor_ids, int64_t* grad_off,
                      int64_t* fac_off_p, int64_t* fac_off_q, int32_t* compressed) {
  if (!c) return ACP_E_INVALID;
  if (b < 0 || b >= static_cast<int32_t>(c->plan.buckets.size()))
    return fail(c, ACP_E_INVALID, "bucket index out of range");
  const acp::BucketPlan& bk = c->plan.buckets[b];
  for (size_t k = 0; k < bk.tids.size(); ++k) {
    if (tensor_ids) tensor_ids[k] = bk.tids[k];
    if (grad_off) grad_off[k] = bk.grad_off[k];
    if (fac_off_p) fac_off_p[k] = bk.fac_off_p[k];
    if (fac_off_q) fac_off_q[k] = bk.fac_off_q[k];
    if (compressed) compressed[k] = c->plan.tensors[bk.tids[k]].compressed ? 1 : 0;
  }
  return ACP_OK;
}

acp_status acp_tensor_info(const acp_ctx* c, int32_t tensor_id, int32_t* compressed, int64_t* n,
                           int64_t* m, int32_t* bucket) {
  if (!c) return ACP_E_INVALID;
  if (tensor_id < 0 || tensor_id >= c->num_tensors) return fail(c, ACP_E_INVALID, "tensor id out of range");
  const acp::TensorPlan& t = c->plan.tensors[tensor_id];
  if (compressed) *compressed = t.compressed ? 1 : 0;
  if (n) *n = t.n;
  if (m) *m = t.m;
  if (bucket) *bucket = t.bucket;
  return ACP_OK;
}

acp_status acp_fusion_groups(const acp_ctx* c, int32_t which, int32_t* group_of, int32_t* num_groups) {
  if (!c) return ACP_E_INVALID;
  if (which != ACP_FACTOR_P && which != ACP_FACTOR_Q) return fail(c, ACP_E_INVALID, "bad factor");
  if (!num_groups) return fail(c, ACP_E_INVALID, "num_groups is NULL");
  const std::vector<acp::TensorPlan>& T = c->plan.tensors;
  // elements tensor t contributes to the step's sent buffer
  auto sent = [&](const acp::TensorPlan& t) -> int64_t {
    if (!t.compressed) return t.numel;
    return (which == ACP_FACTOR_P ? t.n : t.m) * c->plan.rank;
  };
  int64_t total = 0, numel = 0;
  for (const acp::TensorPlan& t : T) {
    total += sent(t);
    numel += t.numel;
  }
  const double rate = static_cast<double>(total) / static_cast<double>(numel);
  const double cap = static_cast<double>(c->plan.cap_bytes) * rate;
  int32_t g = 0;
  int64_t bytes = 0;
  for (size_t k = T.size(); k-- > 0;) {
    if (group_of) group_of[k] = g;
    bytes += sent(T[k]) * 4;
    if (static_cast<double>(bytes) >= cap) {
      ++g;
      bytes = 0;
    }
  }
  *num_groups = g + (bytes > 0 ? 1 : 0);
  return ACP_OK;
}

acp_status acp_init_factor(const acp_ctx* c, int32_t tensor_id, int32_t which, float* host_out,
                           int64_t count) {
  if (!c) return ACP_E_INVALID;
  if (!host_out) return fail(c, ACP_E_INVALID, "host_out is NULL");
  if (tensor_id < 0 || tensor_id >= c->num_tensors) return fail(c, ACP_E_INVALID, "tensor id out of range");
  if (which != ACP_FACTOR_P && which != ACP_FACTOR_Q) return fail(c, ACP_E_INVALID, "bad factor");
  const acp::TensorPlan& t = c->plan.tensors[tensor_id];
  if (t.mat < 0) return fail(c, ACP_E_INVALID, "tensor is not compressed");
  const acp::MatDesc& d = c->plan.mats[t.mat];
  const int64_t need = (which == ACP_FACTOR_P ? t.n : t.m) * c->plan.rank;
  if (count != need) return fail(c, ACP_E_INVALID, "count must be rows * rank");
  const float* src = c->init_fac.data() + (which == ACP_FACTOR_P ? d.p_slot : d.q_slot);
  std::memcpy(host_out, src, static_cast<size_t>(need) * 4);
  return ACP_OK;
}

acp_status acp_compress(acp_ctx* c, int64_t step, int32_t b, const float* grad, float* factor_buf,
                        void* stream) {
  return compress_bucket(c, step, b, grad, factor_buf, stream, nullptr);
}

acp_status acp_compress_noalloc(acp_ctx* c, int64_t step, int32_t b, const float* grad, float* factor_buf,
                                void* stream) {
  if (!c) return ACP_E_INVALID;
  if (b < 0 || b >= static_cast<int32_t>(c->plan.buckets.size()))
    return fail(c, ACP_E_INVALID, "bucket index out of range");
  const acp::BucketPlan& bk = c->plan.buckets[b];
  if (bk.qpart_floats * 4 > acp::kScratchBytes)
    return fail(c, ACP_E_UNSUPPORTED, "bucket " + std::to_string(b) + " needs " +
                                          std::to_string(bk.qpart_floats * 4) +
                                          " bytes of Q-step scratch; the static scratch holds " +
                                          std::to_string(acp::kScratchBytes));
  if (!c->dev) return fail(c, ACP_E_STATE, "state not bound");
  if (!c->scratch) return fail(c, ACP_E_DEVICE, c->scratch_err);
  // the kernels address partial k of a matrix as qpart + MatDesc::qpart + k; the bucket's
  // partials start at qpart_base, so this base puts them at the start of the scratch
  float* base = reinterpret_cast<float*>(reinterpret_cast<uintptr_t>(c->scratch) -
                                         static_cast<uintptr_t>(bk.qpart_base) * sizeof(float));
  return compress_bucket(c, step, b, grad, factor_buf, stream, base);
}

acp_status acp_decompress(acp_ctx* c, int64_t step, int32_t b, const float* agg_factor, float* out,
                          void* stream) {
  if (!c) return ACP_E_INVALID;
  if (c->plan.psgd) return fail(c, ACP_E_UNSUPPORTED, "this context runs Power-SGD (acp_powersgd_*)");
  if (!c->dev) return fail(c, ACP_E_STATE, "state not bound");
  if (b < 0 || b >= static_cast<int32_t>(c->plan.buckets.size()))
    return fail(c, ACP_E_INVALID, "bucket index out of range");
  if (!agg_factor || !out) return fail(c, ACP_E_INVALID, "null buffer");
  if (!aligned16(agg_factor) || !aligned16(out)) return fail(c, ACP_E_INVALID, "buffers must be 16-byte aligned");
  if (c->pending[b] == 0 || c->pending[b] != step)
    return fail(c, ACP_E_STEP, "decompress(" + std::to_string(step) + ") without compress(" +
                                   std::to_string(step) + ")");
  const acp::BucketPlan& bk = c->plan.buckets[b];
  {
    const char* a0 = reinterpret_cast<const char*>(agg_factor);
    const char* o0 = reinterpret_cast<const char*>(out);
    const int64_t fe = (step & 1) ? bk.fac_elems_p : bk.fac_elems_q;
    if (o0 < a0 + fe * 4 && a0 < o0 + bk.grad_elems * 4)
      return fail(c, ACP_E_INVALID, "out overlaps agg_factor");
  }
  const acp_status ds = check_device(c);
  if (ds != ACP_OK) return ds;
  acp::KArgs a = base_args(c);
  a.base = b;
  a.src[0] = agg_factor;
  a.dst[0] = out;
  a.parity = static_cast<int32_t>(step & 1);
  set_form(a, 0, c->deferred[b]);
  bool applied = false;
  RunOpts o;
  o.apply = leading_apply(c, bk.compress[(step + 1) & 1]);
  o.applied = &applied;
  const acp_status st = run(c, bk.decompress[step & 1], a, static_cast<hipStream_t>(stream), o);
  if (st != ACP_OK) return st;
  c->pending[b] = 0;
  c->last_step[b] = step;
  c->applied[b] = applied ? step + 1 : 0;
  return ACP_OK;
}

acp_status acp_compress_all(acp_ctx* c, int64_t step, const float* const* grads,
                            float* const* factor_bufs, void* stream) {
  if (!c) return ACP_E_INVALID;
  if (c->plan.psgd) return fail(c, ACP_E_UNSUPPORTED, "this context runs Power-SGD (acp_powersgd_*)");
  if (!c->dev) return fail(c, ACP_E_STATE, "state not bound");
  if (!grads || !factor_bufs) return fail(c, ACP_E_INVALID, "null pointer array");
  const int32_t nb = static_cast<int32_t>(c->plan.buckets.size());
  for (int32_t b = 0; b < nb; ++b) {
    const acp::BucketPlan& bk = c->plan.buckets[b];
    if (!grads[b] || !factor_bufs[b]) return fail(c, ACP_E_INVALID, "null buffer");
    if (!aligned16(grads[b]) || !aligned16(factor_bufs[b]))
      return fail(c, ACP_E_INVALID, "buffers must be 16-byte aligned");
    if (c->pending[b] != 0 || step != c->last_step[b] + 1)
      return fail(c, ACP_E_STEP, "bucket " + std::to_string(b) + " is not ready for step " +
                                     std::to_string(step));
    const char* g0 = reinterpret_cast<const char*>(grads[b]);
    const char* f0 = reinterpret_cast<const char*>(factor_bufs[b]);
    const int64_t fe = (step & 1) ? bk.fac_elems_p : bk.fac_elems_q;
    if (g0 < f0 + fe * 4 && f0 < g0 + bk.grad_elems * 4)
      return fail(c, ACP_E_INVALID, "factor_buf overlaps grad");
  }
  const acp_status ds = check_device(c);
  if (ds != ACP_OK) return ds;
  for (size_t g = 0; g < c->plan.group_compress.size(); ++g) {
    acp::KArgs a = base_args(c);
    a.base = static_cast<int32_t>(g) * acp::kMaxGroup;
    a.parity = static_cast<int32_t>(step & 1);
    a.step = step;
    for (int32_t i = 0; i < acp::kMaxGroup && a.base + i < nb; ++i) {
      a.src[i] = grads[a.base + i];
      a.dst[i] = factor_bufs[a.base + i];
      set_form(a, i, c->deferred[a.base + i]);
    }
    if (!c->plan.reuse) {
      const acp_status sd = run(c, c->plan.group_draw[g][step & 1], a, static_cast<hipStream_t>(stream));
      if (sd != ACP_OK) return sd;
    }
    // the group's K_APPLY is left out when the previous decompress formed every bucket's factor
    RunOpts o;
    o.skip_apply = true;
    for (int32_t i = 0; i < acp::kMaxGroup && a.base + i < nb; ++i)
      if (c->applied[a.base + i] != step) o.skip_apply = false;
    const acp_status st = run(c, c->plan.group_compress[g][step & 1], a, static_cast<hipStream_t>(stream), o);
    if (st != ACP_OK) return st;
  }
  for (int32_t b = 0; b < nb; ++b) {
    c->pending[b] = step;
    c->deferred[b] = form_after_compress(c, step);
    c->applied[b] = 0;
  }
  return ACP_OK;
}

acp_status acp_decompress_all(acp_ctx* c, int64_t step, const float* const* agg_factors,
                              float* const* outs, void* stream) {
  if (!c) return ACP_E_INVALID;
  if (c->plan.psgd) return fail(c, ACP_E_UNSUPPORTED, "this context runs Power-SGD (acp_powersgd_*)");
  if (!c->dev) return fail(c, ACP_E_STATE, "state not bound");
  if (!agg_factors || !outs) return fail(c, ACP_E_INVALID, "null pointer array");
  const int32_t nb = static_cast<int32_t>(c->plan.buckets.size());
  for (int32_t b = 0; b < nb; ++b) {
    const acp::BucketPlan& bk = c->plan.buckets[b];
    if (!agg_factors[b] || !outs[b]) return fail(c, ACP_E_INVALID, "null buffer");
    if (!aligned16(agg_factors[b]) || !aligned16(outs[b]))
      return fail(c, ACP_E_INVALID, "buffers must be 16-byte aligned");
    if (c->pending[b] != step)
      return fail(c, ACP_E_STEP, "bucket " + std::to_string(b) + " has no compressed step " +
                                     std::to_string(step));
    const char* a0 = reinterpret_cast<const char*>(agg_factors[b]);
    const char* o0 = reinterpret_cast<const char*>(outs[b]);
    const int64_t fe = (step & 1) ? bk.fac_elems_p : bk.fac_elems_q;
    if (o0 < a0 + fe * 4 && a0 < o0 + bk.grad_elems * 4)
      return fail(c, ACP_E_INVALID, "out overlaps agg_factor");
  }
  const acp_status ds = check_device(c);
  if (ds != ACP_OK) return ds;
  std::vector<bool> group_applied(c->plan.group_decompress.size(), false);
  for (size_t g = 0; g < c->plan.group_decompress.size(); ++g) {
    acp::KArgs a = base_args(c);
    a.base = static_cast<int32_t>(g) * acp::kMaxGroup;
    a.parity = static_cast<int32_t>(step & 1);
    for (int32_t i = 0; i < acp::kMaxGroup && a.base + i < nb; ++i) {
      a.src[i] = agg_factors[a.base + i];
      a.dst[i] = outs[a.base + i];
      set_form(a, i, c->deferred[a.base + i]);
    }
    bool applied = false;
    RunOpts o;
    o.apply = leading_apply(c, c->plan.group_compress[g][(step + 1) & 1]);
    o.applied = &applied;
    const acp_status st = run(c, c->plan.group_decompress[g][step & 1], a, static_cast<hipStream_t>(stream), o);
    if (st != ACP_OK) return st;
    group_applied[g] = applied;
  }
  for (int32_t b = 0; b < nb; ++b) {
    c->pending[b] = 0;
    c->last_step[b] = step;
    c->applied[b] = group_applied[b / acp::kMaxGroup] ? step + 1 : 0;
  }
  return ACP_OK;
}

acp_status acp_powersgd_p(acp_ctx* c, int64_t step, int32_t b, const float* grad, float* p_buf,
                          void* stream) {
  if (!c) return ACP_E_INVALID;
  acp_status st = psgd_ready(c, step, b, 0);
  if (st != ACP_OK) return st;
  if (!grad || !p_buf) return fail(c, ACP_E_INVALID, "null buffer");
  if (!aligned16(grad) || !aligned16(p_buf)) return fail(c, ACP_E_INVALID, "buffers must be 16-byte aligned");
  const acp::BucketPlan& bk = c->plan.buckets[b];
  if (overlaps(grad, bk.grad_elems, p_buf, bk.fac_elems_p)) return fail(c, ACP_E_INVALID, "p_buf overlaps grad");
  if ((st = check_device(c)) != ACP_OK) return st;
  if ((st = psgd_p_bucket(c, step, b, grad, p_buf, static_cast<hipStream_t>(stream))) != ACP_OK) return st;
  c->pending[b] = step;
  c->phase[b] = 1;
  return ACP_OK;
}

acp_status acp_powersgd_q(acp_ctx* c, int64_t step, int32_t b, const float* grad, const float* p_agg,
                          float* q_buf, void* stream) {
  if (!c) return ACP_E_INVALID;
  acp_status st = psgd_ready(c, step, b, 1);
  if (st != ACP_OK) return st;
  if (!grad || !p_agg || !q_buf) return fail(c, ACP_E_INVALID, "null buffer");
  if (!aligned16(grad) || !aligned16(p_agg) || !aligned16(q_buf))
    return fail(c, ACP_E_INVALID, "buffers must be 16-byte aligned");
  const acp::BucketPlan& bk = c->plan.buckets[b];
  if (overlaps(q_buf, bk.fac_elems_q, grad, bk.grad_elems) || overlaps(q_buf, bk.fac_elems_q, p_agg, bk.fac_elems_p))
    return fail(c, ACP_E_INVALID, "q_buf overlaps grad or p_agg");
  if ((st = check_device(c)) != ACP_OK) return st;
  if ((st = psgd_q_bucket(c, b, grad, p_agg, q_buf, static_cast<hipStream_t>(stream))) != ACP_OK) return st;
  c->phase[b] = 2;
  c->deferred[b] = c->plan.ef ? kHoldsF : kExplicit;
  return ACP_OK;
}

acp_status acp_powersgd_decompress(acp_ctx* c, int64_t step, int32_t b, const float* q_agg, float* out,
                                   void* stream) {
  if (!c) return ACP_E_INVALID;
  acp_status st = psgd_ready(c, step, b, 2);
  if (st != ACP_OK) return st;
  if (!q_agg || !out) return fail(c, ACP_E_INVALID, "null buffer");
  if (!aligned16(q_agg) || !aligned16(out)) return fail(c, ACP_E_INVALID, "buffers must be 16-byte aligned");
  const acp::BucketPlan& bk = c->plan.buckets[b];
  if (overlaps(out, bk.grad_elems, q_agg, bk.fac_elems_q)) return fail(c, ACP_E_INVALID, "out overlaps q_agg");
  if ((st = check_device(c)) != ACP_OK) return st;
  acp::KArgs a = base_args(c);
  a.copy_only = 1;
  a.base = b;
  a.src[0] = q_agg;
  a.dst[0] = out;
  a.parity = 0;
  set_form(a, 0, c->deferred[b]);
  if ((st = run(c, bk.decompress[0], a, static_cast<hipStream_t>(stream), RunOpts{true})) != ACP_OK) return st;
  c->pending[b] = 0;
  c->phase[b] = 0;
  c->last_step[b] = step;
  return ACP_OK;
}

acp_status acp_powersgd_p_all(acp_ctx* c, int64_t step, const float* const* grads, float* const* p_bufs,
                              void* stream) {
  if (!c) return ACP_E_INVALID;
  if (!grads || !p_bufs) return fail(c, ACP_E_INVALID, "null pointer array");
  const int32_t nb = static_cast<int32_t>(c->plan.buckets.size());
  for (int32_t b = 0; b < nb; ++b) {
    const acp_status st = psgd_ready(c, step, b, 0);
    if (st != ACP_OK) return st;
    const acp::BucketPlan& bk = c->plan.buckets[b];
    if (!grads[b] || !p_bufs[b]) return fail(c, ACP_E_INVALID, "null buffer");
    if (!aligned16(grads[b]) || !aligned16(p_bufs[b])) return fail(c, ACP_E_INVALID, "buffers must be 16-byte aligned");
    if (overlaps(grads[b], bk.grad_elems, p_bufs[b], bk.fac_elems_p)) return fail(c, ACP_E_INVALID, "p_buf overlaps grad");
  }
  acp_status st = check_device(c);
  if (st != ACP_OK) return st;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  for (size_t g = 0; g < c->plan.group_compress.size(); ++g) {
    acp::KArgs a = base_args(c), m = base_args(c);
    a.base = m.base = static_cast<int32_t>(g) * acp::kMaxGroup;
    a.parity = m.parity = 1;
    m.ef = 0;
    for (int32_t i = 0; i < acp::kMaxGroup && a.base + i < nb; ++i) {
      a.src[i] = grads[a.base + i];
      set_form(a, i, c->deferred[a.base + i]);
      m.src[i] = psgd_source(c, a.base + i, grads[a.base + i]);
      m.dst[i] = p_bufs[a.base + i];
    }
    if ((st = run(c, c->plan.group_psgd_image[g], a, s)) != ACP_OK) return st;
    if ((st = run(c, c->plan.group_compress[g][1], m, s)) != ACP_OK) return st;
  }
  for (int32_t b = 0; b < nb; ++b) {
    c->pending[b] = step;
    c->phase[b] = 1;
  }
  return ACP_OK;
}

acp_status acp_powersgd_q_all(acp_ctx* c, int64_t step, const float* const* grads, const float* const* p_aggs,
                              float* const* q_bufs, void* stream) {
  if (!c) return ACP_E_INVALID;
  if (!grads || !p_aggs || !q_bufs) return fail(c, ACP_E_INVALID, "null pointer array");
  const int32_t nb = static_cast<int32_t>(c->plan.buckets.size());
  for (int32_t b = 0; b < nb; ++b) {
    const acp_status st = psgd_ready(c, step, b, 1);
    if (st != ACP_OK) return st;
    const acp::BucketPlan& bk = c->plan.buckets[b];
    if (!grads[b] || !p_aggs[b] || !q_bufs[b]) return fail(c, ACP_E_INVALID, "null buffer");
    if (!aligned16(grads[b]) || !aligned16(p_aggs[b]) || !aligned16(q_bufs[b]))
      return fail(c, ACP_E_INVALID, "buffers must be 16-byte aligned");
    if (overlaps(q_bufs[b], bk.fac_elems_q, grads[b], bk.grad_elems) ||
        overlaps(q_bufs[b], bk.fac_elems_q, p_aggs[b], bk.fac_elems_p))
      return fail(c, ACP_E_INVALID, "q_buf overlaps grad or p_agg");
  }
  acp_status st = check_device(c);
  if (st != ACP_OK) return st;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  for (size_t g = 0; g < c->plan.group_compress.size(); ++g) {
    acp::KArgs a = base_args(c), m = base_args(c);
    a.base = m.base = static_cast<int32_t>(g) * acp::kMaxGroup;
    a.parity = m.parity = 0;
    m.ef = 0;
    for (int32_t i = 0; i < acp::kMaxGroup && a.base + i < nb; ++i) {
      a.src[i] = p_aggs[a.base + i];
      m.src[i] = psgd_source(c, a.base + i, grads[a.base + i]);
      m.dst[i] = q_bufs[a.base + i];
    }
    if ((st = run(c, c->plan.group_psgd_fact[g], a, s)) != ACP_OK) return st;
    if ((st = run(c, c->plan.group_compress[g][0], m, s)) != ACP_OK) return st;
  }
  for (int32_t b = 0; b < nb; ++b) {
    c->phase[b] = 2;
    c->deferred[b] = c->plan.ef ? kHoldsF : kExplicit;
  }
  return ACP_OK;
}

acp_status acp_powersgd_decompress_all(acp_ctx* c, int64_t step, const float* const* q_aggs, float* const* outs,
                                       void* stream) {
  if (!c) return ACP_E_INVALID;
  if (!q_aggs || !outs) return fail(c, ACP_E_INVALID, "null pointer array");
  const int32_t nb = static_cast<int32_t>(c->plan.buckets.size());
  for (int32_t b = 0; b < nb; ++b) {
    const acp_status st = psgd_ready(c, step, b, 2);
    if (st != ACP_OK) return st;
    const acp::BucketPlan& bk = c->plan.buckets[b];
    if (!q_aggs[b] || !outs[b]) return fail(c, ACP_E_INVALID, "null buffer");
    if (!aligned16(q_aggs[b]) || !aligned16(outs[b])) return fail(c, ACP_E_INVALID, "buffers must be 16-byte aligned");
    if (overlaps(outs[b], bk.grad_elems, q_aggs[b], bk.fac_elems_q)) return fail(c, ACP_E_INVALID, "out overlaps q_agg");
  }
  acp_status st = check_device(c);
  if (st != ACP_OK) return st;
  for (size_t g = 0; g < c->plan.group_decompress.size(); ++g) {
    acp::KArgs a = base_args(c);
    a.copy_only = 1;
    a.base = static_cast<int32_t>(g) * acp::kMaxGroup;
    a.parity = 0;
    for (int32_t i = 0; i < acp::kMaxGroup && a.base + i < nb; ++i) {
      a.src[i] = q_aggs[a.base + i];
      a.dst[i] = outs[a.base + i];
      set_form(a, i, c->deferred[a.base + i]);
    }
    if ((st = run(c, c->plan.group_decompress[g][0], a, static_cast<hipStream_t>(stream), RunOpts{true})) != ACP_OK)
      return st;
  }
  for (int32_t b = 0; b < nb; ++b) {
    c->pending[b] = 0;
    c->phase[b] = 0;
    c->last_step[b] = step;
  }
  return ACP_OK;
}

acp_status acp_error(const acp_ctx* c, int32_t b, float* e_out, void* stream) {
  if (!c) return ACP_E_INVALID;
  if (!c->dev) return fail(c, ACP_E_STATE, "state not bound");
  if (!c->plan.ef) return fail(c, ACP_E_UNSUPPORTED, "no error feedback in this context");
  if (b < 0 || b >= static_cast<int32_t>(c->plan.buckets.size()))
    return fail(c, ACP_E_INVALID, "bucket index out of range");
  if (!e_out || !aligned16(e_out)) return fail(c, ACP_E_INVALID, "e_out must be a 16-byte aligned pointer");
  if (c->plan.psgd && c->phase[b] == 1)
    return fail(c, ACP_E_STEP, "between the halves of a Power-SGD step the E arena holds M + E");
  const acp_status ds = check_device(c);
  if (ds != ACP_OK) return ds;
  acp::KArgs a = base_args(c);
  a.base = b;
  a.dst[0] = e_out;
  set_form(a, 0, c->deferred[b]);
  return run(c, c->plan.buckets[b].emat, a, static_cast<hipStream_t>(stream));
}

acp_status acp_factor(const acp_ctx* c, int32_t tensor_id, int32_t which, float* dev_out, void* stream) {
  if (!c) return ACP_E_INVALID;
  if (!c->dev) return fail(c, ACP_E_STATE, "state not bound");
  if (tensor_id < 0 || tensor_id >= c->num_tensors) return fail(c, ACP_E_INVALID, "tensor id out of range");
  if (which != ACP_FACTOR_P && which != ACP_FACTOR_Q) return fail(c, ACP_E_INVALID, "bad factor");
  if (!dev_out) return fail(c, ACP_E_INVALID, "dev_out is NULL");
  const acp::TensorPlan& t = c->plan.tensors[tensor_id];
  if (t.mat < 0) return fail(c, ACP_E_INVALID, "tensor is not compressed");
  const int64_t step = c->last_step[t.bucket];
  if (step < 1) return fail(c, ACP_E_STEP, "no completed step");
  const acp::MatDesc& d = c->plan.mats[t.mat];
  const bool odd = (step & 1) != 0 && !c->plan.psgd;  // a Power-SGD step ends like a Q-step
  int64_t slot, rows;
  if (which == ACP_FACTOR_P) {
    slot = odd ? d.p_slot : d.ph_slot;
    rows = t.n;
  } else {
    slot = odd ? d.qh_slot : d.q_slot;
    rows = t.m;
  }
  const acp_status ds = check_device(c);
  if (ds != ACP_OK) return ds;
  const hipError_t e = hipMemcpyAsync(dev_out, c->dev + c->plan.off_fac + slot * 4,
                                      rows * c->plan.rank * 4, hipMemcpyDeviceToDevice,
                                      static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(c, ACP_E_DEVICE, std::string("copy failed: ") + hipGetErrorString(e));
  return ACP_OK;
}

acp_status acp_checkpoint_bytes(const acp_ctx* c, int64_t* bytes) {
  if (!c || !bytes) return fail(c, ACP_E_INVALID, "null argument");
  const int64_t nb = static_cast<int64_t>(c->plan.buckets.size());
  *bytes = static_cast<int64_t>(sizeof(CkptHeader)) + nb * 16 + checkpoint_payload(c->plan);
  return ACP_OK;
}

acp_status acp_get_state(const acp_ctx* c, void* host_buf, int64_t bytes) {
  if (!c) return ACP_E_INVALID;
  if (!c->dev) return fail(c, ACP_E_STATE, "state not bound");
  if (!host_buf) return fail(c, ACP_E_INVALID, "host_buf is NULL");
  int64_t need = 0;
  acp_checkpoint_bytes(c, &need);
  if (bytes < need) return fail(c, ACP_E_INVALID, "host buffer too small");
  for (int64_t p : c->pending)
    if (p) return fail(c, ACP_E_STEP, "a bucket is between compress and decompress");
  const acp_status ds = check_device(c);
  if (ds != ACP_OK) return ds;
  const acp::Plan& p = c->plan;
  CkptHeader h{kMagic, kVersion, c->num_tensors, p.rank, p.cap_bytes, c->world, c->flags,
               static_cast<int64_t>(p.buckets.size()), static_cast<int64_t>(c->seed),
               p.e_floats, p.fac_floats, p.w_doubles};
  uint8_t* o = static_cast<uint8_t*>(host_buf);
  std::memcpy(o, &h, sizeof(h));
  o += sizeof(h);
  for (size_t b = 0; b < p.buckets.size(); ++b) {
    const int64_t rec[2] = {c->last_step[b], static_cast<int64_t>(c->deferred[b])};
    std::memcpy(o, rec, 16);
    o += 16;
  }
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess && p.e_floats) e = hipMemcpy(o, c->dev + p.off_e, p.e_floats * 4, hipMemcpyDeviceToHost);
  o += p.e_floats * 4;
  if (e == hipSuccess && p.fac_floats) e = hipMemcpy(o, c->dev + p.off_fac, p.fac_floats * 4, hipMemcpyDeviceToHost);
  o += p.fac_floats * 4;
  if (e == hipSuccess && p.w_doubles) e = hipMemcpy(o, c->dev + p.off_w, p.w_doubles * 8, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return fail(c, ACP_E_DEVICE, std::string("state download failed: ") + hipGetErrorString(e));
  return ACP_OK;
}

acp_status acp_set_state(acp_ctx* c, const void* host_buf, int64_t bytes) {
  if (!c) return ACP_E_INVALID;
  if (!c->dev) return fail(c, ACP_E_STATE, "state not bound");
  if (!host_buf) return fail(c, ACP_E_INVALID, "host_buf is NULL");
  int64_t need = 0;
  acp_checkpoint_bytes(c, &need);
  if (bytes < need) return fail(c, ACP_E_STATE, "checkpoint too small");
  for (int64_t p : c->pending)
    if (p) return fail(c, ACP_E_STEP, "a bucket is between compress and decompress");
  const acp::Plan& p = c->plan;
  CkptHeader h{};
  std::memcpy(&h, host_buf, sizeof(h));
  if (h.magic != kMagic || h.version != kVersion || h.num_tensors != c->num_tensors ||
      h.rank != p.rank || h.cap != p.cap_bytes || h.world != c->world ||
      h.flags != static_cast<int64_t>(c->flags) || h.nbuckets != static_cast<int64_t>(p.buckets.size()) ||
      h.seed != static_cast<int64_t>(c->seed) || h.e_floats != p.e_floats ||
      h.fac_floats != p.fac_floats || h.w_doubles != p.w_doubles)
    return fail(c, ACP_E_STATE, "checkpoint does not match this context");
  const acp_status ds = check_device(c);
  if (ds != ACP_OK) return ds;
  const uint8_t* i = static_cast<const uint8_t*>(host_buf) + sizeof(h);
  std::vector<int64_t> steps(p.buckets.size());
  std::vector<uint8_t> defr(p.buckets.size());
  for (size_t b = 0; b < p.buckets.size(); ++b) {
    int64_t rec[2];
    std::memcpy(rec, i, 16);
    i += 16;
    if (rec[0] < 0 || rec[1] < 0 || rec[1] > kHoldsX) return fail(c, ACP_E_STATE, "corrupt checkpoint");
    steps[b] = rec[0];
    defr[b] = static_cast<uint8_t>(rec[1]);
  }
  hipError_t e = hipDeviceSynchronize();
  if (e == hipSuccess && p.e_floats) e = hipMemcpy(c->dev + p.off_e, i, p.e_floats * 4, hipMemcpyHostToDevice);
  i += p.e_floats * 4;
  if (e == hipSuccess && p.fac_floats) e = hipMemcpy(c->dev + p.off_fac, i, p.fac_floats * 4, hipMemcpyHostToDevice);
  i += p.fac_floats * 4;
  if (e == hipSuccess && p.w_doubles) e = hipMemcpy(c->dev + p.off_w, i, p.w_doubles * 8, hipMemcpyHostToDevice);
  if (e != hipSuccess) return fail(c, ACP_E_DEVICE, std::string("state upload failed: ") + hipGetErrorString(e));
  c->last_step = steps;
  c->deferred = defr;
  c->applied.assign(p.buckets.size(), 0);
  return ACP_OK;
}

acp_status acp_profile_start(acp_ctx* c, int32_t kernel_family, int32_t max_launches) {
  if (!c) return ACP_E_INVALID;
  if (kernel_family < ACP_KERNEL_P_STEP || kernel_family > ACP_KERNEL_ORTH)
    return fail(c, ACP_E_INVALID, "unknown kernel family");
  if (max_launches < 1 || max_launches > (1 << 20)) return fail(c, ACP_E_INVALID, "bad max_launches");
  if (!c->dev) return fail(c, ACP_E_STATE, "state not bound");
  if (c->prof_family != 0) return fail(c, ACP_E_STATE, "profiling already active");
  const acp_status ds = check_device(c);
  if (ds != ACP_OK) return ds;
  c->prof_events.assign(2 * static_cast<size_t>(max_launches), nullptr);
  for (hipEvent_t& ev : c->prof_events) {
    if (hipEventCreate(&ev) != hipSuccess) {
      for (hipEvent_t& e2 : c->prof_events)
        if (e2) (void)hipEventDestroy(e2);
      c->prof_events.clear();
      return fail(c, ACP_E_DEVICE, "hipEventCreate failed");
    }
  }
  c->prof_family = kernel_family;
  c->prof_used = 0;
  c->prof_bytes = 0.0;
  return ACP_OK;
}

acp_status acp_profile_stop(acp_ctx* c, int64_t* launches, double* seconds, double* alg_bytes) {
  if (!c) return ACP_E_INVALID;
  if (c->prof_family == 0) return fail(c, ACP_E_STATE, "profiling not active");
  double total_ms = 0.0;
  acp_status st = ACP_OK;
  for (int64_t i = 0; i < c->prof_used; ++i) {
    float ms = 0.f;
    if (hipEventSynchronize(c->prof_events[2 * i + 1]) != hipSuccess ||
        hipEventElapsedTime(&ms, c->prof_events[2 * i], c->prof_events[2 * i + 1]) != hipSuccess) {
      st = fail(c, ACP_E_DEVICE, "reading profile events failed");
      break;
    }
    total_ms += ms;
  }
  for (hipEvent_t& ev : c->prof_events)
    if (ev) (void)hipEventDestroy(ev);
  if (launches) *launches = c->prof_used;
  if (seconds) *seconds = total_ms * 1e-3;
  if (alg_bytes) *alg_bytes = c->prof_bytes;
  c->prof_events.clear();
  c->prof_family = 0;
  c->prof_used = 0;
  c->prof_bytes = 0.0;
  return st;
}

const char* acp_last_error(const acp_ctx* c) { return c ? c->err.c_str() : "null context"; }

void acp_destroy(acp_ctx* c) {
  if (!c) return;
  for (hipEvent_t& ev : c->prof_events)
    if (ev) (void)hipEventDestroy(ev);
  release_side(c);
  delete c;
}

}  // extern "C"
