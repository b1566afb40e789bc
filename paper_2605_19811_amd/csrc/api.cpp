// C ABI of the LionMuon step (declared in include/lionmuon.h): validation,
// the cache of uploaded plans, the library-owned workspace, phase timing and
// the launch sequence of Algorithm 1 on one stream.
#include <hip/hip_runtime_api.h>

#include <cmath>
#include <cstring>
#include <deque>
#include <list>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"
#include "lionmuon.h"
#include "plan.h"

namespace {

using lm::Plan;
using lm::Status;
using lm::TensorIn;

thread_local std::string g_last_error;

lm_status fail(lm_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

lm_status to_c(Status s) { return static_cast<lm_status>(static_cast<int>(s)); }

lm_status hip_fail(hipError_t e, const char* what) {
  return fail(LM_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// ---------------------------------------------------------------------------
// Device shape
// ---------------------------------------------------------------------------
// Compute units and XCDs of a device, read once per device. Without a
// device (host-only queries on a machine with no GPU) a full MI355X is
// assumed: 256 CUs in 8 XCDs.
std::mutex g_chip_mu;
std::vector<std::pair<int, lm::ChipShape>> g_chips;

lm::ChipShape chip_of(int device) {
  std::lock_guard<std::mutex> lock(g_chip_mu);
  for (const auto& c : g_chips)
    if (c.first == device) return c.second;
  lm::ChipShape chip;
  int cus = 0, xccs = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) == hipSuccess &&
      cus > 0) {
    chip.cus = cus;
    if (hipDeviceGetAttribute(&xccs, hipDeviceAttributeNumberOfXccs, device) != hipSuccess ||
        xccs < 1)
      xccs = 1;
    chip.xcds = std::min(xccs, lm::kMaxXcds);
    if (chip.cus < chip.xcds) chip.xcds = chip.cus;
  } else {
    (void)hipGetLastError();
  }
  g_chips.push_back({device, chip});
  return chip;
}

// Shape of the current device, or the MI355X default when there is none.
lm::ChipShape current_chip() {
  int device = 0;
  if (hipGetDevice(&device) != hipSuccess) {
    (void)hipGetLastError();
    return lm::ChipShape();
  }
  return chip_of(device);
}

// ---------------------------------------------------------------------------
// Pinned staging ring
// ---------------------------------------------------------------------------
// Host-to-device copies of per-call binding tables are staged through one
// pinned ring. A region is handed out again only after the event recorded
// behind its copy has completed, which a host that runs no further ahead of
// the device than the ring's capacity never waits for.
struct StagingRing {
  uint8_t* host = nullptr;
  size_t cap = 0;
  uint64_t head = 0;                 // bytes handed out so far (monotonic)
  struct Region {
    uint64_t start, end;
    hipEvent_t done;
  };
  std::deque<Region> inflight;       // oldest first
  std::vector<hipEvent_t> pool;
};
StagingRing g_ring;

// ---------------------------------------------------------------------------
// Uploaded plans
// ---------------------------------------------------------------------------
// One plan per (device, step kind, NS element size, scaling, and the
// tensors' shapes, flags and 16-byte alignment). Its descriptor tables live in
// one device allocation, filled once from a pinned host copy on the stream of
// the call that created the plan. The same allocation holds the plan's
// binding table (one TensorPtrs per input tensor), rewritten on the call's
// stream whenever a call brings other tensor addresses than the previous
// call of the plan.
struct DevicePlan {
  Plan plan;
  int device = -1;
  std::vector<uint8_t> key;
  void* dev = nullptr;
  void* host = nullptr;             // pinned staging copy of the tables
  hipEvent_t last_use = nullptr;    // recorded after the last call that used the plan
  hipStream_t last_stream = nullptr;
  std::vector<lm::TensorPtrs> bound;   // addresses the device binding holds
  lm::TensorPtrs* d_bind = nullptr;
  lm::LionTensor* d_lion = nullptr;
  int32_t* d_lion_start = nullptr;
  lm::MuonMat* d_mats = nullptr;
  int32_t* d_prep_start = nullptr;
  lm::SrBlock* d_sr_tab = nullptr;
  int32_t* d_rd_start = nullptr;
  int32_t* d_tensor_mat = nullptr;
  lm::GemmTask* d_tasks[2][4] = {};   // [precision][gram, poly, apply, apply tail]
  lm::XcdSplit* d_splits = nullptr;   // [precision * 4 + list]

  ~DevicePlan() {
    if (last_use) (void)hipEventDestroy(last_use);
    if (dev) (void)hipFree(dev);
    if (host) (void)hipHostFree(host);
  }
};

constexpr size_t kMaxPlans = 16;
std::mutex g_mu;                                      // plans, workspace, profiling, ring
std::list<std::shared_ptr<DevicePlan>> g_plans;       // most recent first

// The library-owned workspace of a device. Calls that use it are serialised
// on the host by g_mu, but their kernels run on the callers' streams: a call
// on another stream than the previous user's first waits (on the device) for
// the event recorded after that user's work.
struct OwnedWorkspace {
  int device = -1;
  void* ptr = nullptr;
  size_t bytes = 0;
  hipEvent_t done = nullptr;       // recorded after the last call that used it
  hipStream_t last = nullptr;      // that call's stream
};
std::vector<OwnedWorkspace> g_ws;

// Phase timing (never in the no-allocation entry point, which creates no
// events)
bool g_prof = false;
bool g_prof_suppressed = false;
struct PendingEvent {
  int phase;
  hipEvent_t start, stop;
};
std::vector<PendingEvent> g_pending;
std::vector<hipEvent_t> g_event_pool;
lm_phase_times g_times{};

hipError_t get_event(hipEvent_t* e) {
  if (!g_event_pool.empty()) {
    *e = g_event_pool.back();
    g_event_pool.pop_back();
    return hipSuccess;
  }
  // device-scope only: a system-scope release on every phase boundary costs
  // several microseconds per event, and the timestamps are read back only
  // after the stream has been synchronised
  return hipEventCreateWithFlags(e, hipEventDisableSystemFence);
}

void append_key(std::vector<uint8_t>* k, const void* p, size_t n) {
  const uint8_t* b = static_cast<const uint8_t*>(p);
  k->insert(k->end(), b, b + n);
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

template <typename T>
void place(std::vector<T>& v, size_t* off, std::vector<std::pair<size_t, std::pair<const void*, size_t>>>* parts) {
  parts->push_back({*off, {v.data(), v.size() * sizeof(T)}});
  *off = align256(*off + v.size() * sizeof(T));
}

// The call's tensor addresses, one entry per input tensor.
std::vector<lm::TensorPtrs> binding_of(const TensorIn* x, int32_t n) {
  std::vector<lm::TensorPtrs> b(size_t(n > 0 ? n : 0));
  for (int32_t i = 0; i < n; ++i) {
    b[size_t(i)].w = x[i].w;
    b[size_t(i)].g = x[i].g;
    b[size_t(i)].m = x[i].m;
    b[size_t(i)].v = (x[i].flags & lm::kFlagAdamW) ? x[i].v : nullptr;
  }
  return b;
}

bool same_binding(const std::vector<lm::TensorPtrs>& a, const std::vector<lm::TensorPtrs>& b) {
  return a.size() == b.size() &&
         (a.empty() || std::memcmp(a.data(), b.data(), a.size() * sizeof(lm::TensorPtrs)) == 0);
}

// Copy `bytes` from host memory to device memory `dst` on `stream` through
// the pinned ring (the source may be reused as soon as this returns).
lm_status stage_upload(void* dst, const void* src, size_t bytes, hipStream_t stream) {
  StagingRing& r = g_ring;
  hipError_t e = hipSuccess;
  const size_t need = (bytes + 63) & ~size_t(63);
  if (need > r.cap) {
    // grow: wait for every staged copy, then replace the ring
    for (auto& reg : r.inflight) {
      (void)hipEventSynchronize(reg.done);
      r.pool.push_back(reg.done);
    }
    r.inflight.clear();
    if (r.host) (void)hipHostFree(r.host);
    r.host = nullptr;
    r.cap = 0;
    size_t cap = size_t(1) << 20;
    while (cap < 4 * need) cap <<= 1;
    void* h = nullptr;
    e = hipHostMalloc(&h, cap, hipHostMallocPortable);
    if (e != hipSuccess) return fail(LM_ERR_OUT_OF_MEMORY, "staging ring: hipHostMalloc failed");
    r.host = static_cast<uint8_t*>(h);
    r.cap = cap;
  }
  uint64_t s = r.head;
  if (s % r.cap + need > r.cap) s += r.cap - s % r.cap;   // no region straddles the end
  while (!r.inflight.empty() && r.inflight.front().start + r.cap < s + need) {
    e = hipEventSynchronize(r.inflight.front().done);
    if (e != hipSuccess) return hip_fail(e, "staging ring: hipEventSynchronize");
    r.pool.push_back(r.inflight.front().done);
    r.inflight.pop_front();
  }
  uint8_t* h = r.host + s % r.cap;
  std::memcpy(h, src, bytes);
  e = hipMemcpyAsync(dst, h, bytes, hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) return hip_fail(e, "binding upload: hipMemcpyAsync");
  hipEvent_t ev = nullptr;
  if (!r.pool.empty()) {
    ev = r.pool.back();
    r.pool.pop_back();
  } else {
    e = hipEventCreateWithFlags(&ev, hipEventDisableTiming | hipEventDisableSystemFence);
    if (e != hipSuccess) return hip_fail(e, "staging ring: hipEventCreate");
  }
  e = hipEventRecord(ev, stream);
  if (e != hipSuccess) {
    r.pool.push_back(ev);
    return hip_fail(e, "staging ring: hipEventRecord");
  }
  r.inflight.push_back({s, s + need, ev});
  r.head = s + need;
  return LM_OK;
}

// Cache key of a list signature: device, step kind, NS precision and
// scaling, then each tensor's shape, flags and alignment class.
std::vector<uint8_t> plan_key(int device, const TensorIn* x, int32_t n, lm::StepKind kind,
                              lm::NsPrecision prec, bool rms02) {
  std::vector<uint8_t> key;
  key.reserve(size_t(n) * 24 + 32);
  const int32_t hdr[5] = {device, static_cast<int32_t>(kind), prec.all_fp32 ? 1 : 0,
                          prec.bf16_min_side, rms02 ? 1 : 0};
  append_key(&key, hdr, sizeof(hdr));
  for (int32_t i = 0; i < n; ++i) {
    const int64_t dims[2] = {x[i].rows, x[i].cols};
    const uint32_t fa[2] = {x[i].flags, lm::align_class(x[i])};
    append_key(&key, dims, sizeof(dims));
    append_key(&key, fa, sizeof(fa));
  }
  return key;
}

// Device image of a plan's tables and binding: one byte block, each table
// 256-byte aligned at its offset.
struct TableImage {
  std::vector<uint8_t> bytes;
  size_t o_bind = 0, o_lion = 0, o_lion_start = 0, o_mats = 0, o_prep = 0, o_sr = 0, o_rd = 0,
         o_tm = 0, o_splits = 0;
  size_t o_tasks[2][4] = {};
};

void pack_tables(Plan& p, std::vector<lm::TensorPtrs>& bind, TableImage* img) {
  std::vector<std::pair<size_t, std::pair<const void*, size_t>>> parts;
  size_t off = 0;
  img->o_bind = off;       place(bind, &off, &parts);
  img->o_lion = off;       place(p.lion, &off, &parts);
  img->o_lion_start = off; place(p.lion_block_start, &off, &parts);
  img->o_mats = off;       place(p.mats, &off, &parts);
  img->o_prep = off;       place(p.prep_start, &off, &parts);
  img->o_sr = off;         place(p.sr_tab, &off, &parts);
  img->o_rd = off;         place(p.rd_start, &off, &parts);
  img->o_tm = off;         place(p.tensor_mat, &off, &parts);
  std::vector<lm::XcdSplit> splits;
  for (int pr = 0; pr < 2; ++pr) {
    img->o_tasks[pr][0] = off; place(p.gram[pr], &off, &parts);
    img->o_tasks[pr][1] = off; place(p.poly[pr], &off, &parts);
    img->o_tasks[pr][2] = off; place(p.apply[pr], &off, &parts);
    img->o_tasks[pr][3] = off; place(p.apply_tail[pr], &off, &parts);
    splits.push_back(p.gram_split[pr]);
    splits.push_back(p.poly_split[pr]);
    splits.push_back(p.apply_split[pr]);
    splits.push_back(p.apply_tail_split[pr]);
  }
  img->o_splits = off;     place(splits, &off, &parts);
  img->bytes.assign(std::max<size_t>(off, 256), 0);
  for (const auto& part : parts)
    if (part.second.second)
      std::memcpy(img->bytes.data() + part.first, part.second.first, part.second.second);
}

// Point a plan's device table pointers into the image placed at `base`.
void point_tables(DevicePlan* dp, uint8_t* base, const TableImage& img) {
  dp->d_bind = reinterpret_cast<lm::TensorPtrs*>(base + img.o_bind);
  dp->d_lion = reinterpret_cast<lm::LionTensor*>(base + img.o_lion);
  dp->d_lion_start = reinterpret_cast<int32_t*>(base + img.o_lion_start);
  dp->d_mats = reinterpret_cast<lm::MuonMat*>(base + img.o_mats);
  dp->d_prep_start = reinterpret_cast<int32_t*>(base + img.o_prep);
  dp->d_sr_tab = reinterpret_cast<lm::SrBlock*>(base + img.o_sr);
  dp->d_rd_start = reinterpret_cast<int32_t*>(base + img.o_rd);
  dp->d_tensor_mat = reinterpret_cast<int32_t*>(base + img.o_tm);
  for (int pr = 0; pr < 2; ++pr)
    for (int st4 = 0; st4 < 4; ++st4)
      dp->d_tasks[pr][st4] = reinterpret_cast<lm::GemmTask*>(base + img.o_tasks[pr][st4]);
  dp->d_splits = reinterpret_cast<lm::XcdSplit*>(base + img.o_splits);
}

// Find or build the plan of this list signature and make its tables and
// binding ready on `stream`: the stream first waits (on the device) for the
// plan's last user when that ran on another stream, and the binding is
// rewritten when the call's addresses differ from those it holds.
lm_status get_plan(const TensorIn* x, int32_t n, lm::StepKind kind, lm::NsPrecision prec,
                   bool rms02, hipStream_t stream, std::shared_ptr<DevicePlan>* out) {
  int device = 0;
  hipError_t e = hipGetDevice(&device);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::vector<uint8_t> key = plan_key(device, x, n, kind, prec, rms02);
  std::vector<lm::TensorPtrs> bind = binding_of(x, n);
  for (auto it = g_plans.begin(); it != g_plans.end(); ++it) {
    if ((*it)->key == key) {
      g_plans.splice(g_plans.begin(), g_plans, it);
      DevicePlan& dp = *g_plans.front();
      if (dp.last_use && dp.last_stream != stream) {
        e = hipStreamWaitEvent(stream, dp.last_use, 0);
        if (e != hipSuccess) return hip_fail(e, "hipStreamWaitEvent");
      }
      if (!same_binding(dp.bound, bind)) {
        lm_status s = stage_upload(dp.d_bind, bind.data(), bind.size() * sizeof(lm::TensorPtrs),
                                   stream);
        if (s != LM_OK) return s;
        dp.bound.swap(bind);
      }
      *out = g_plans.front();
      return LM_OK;
    }
  }
  auto dp = std::make_shared<DevicePlan>();
  dp->device = device;
  dp->key = std::move(key);
  std::string err;
  Status st = lm::build_plan(x, n, kind, prec, rms02, chip_of(device), &dp->plan, &err);
  if (st != Status::kOk) return fail(to_c(st), err);
  TableImage img;
  pack_tables(dp->plan, bind, &img);
  const size_t total = img.bytes.size();
  e = hipMalloc(&dp->dev, total);
  if (e != hipSuccess) return fail(LM_ERR_OUT_OF_MEMORY, "plan tables: hipMalloc failed");
  e = hipHostMalloc(&dp->host, total, hipHostMallocDefault);
  if (e != hipSuccess) return fail(LM_ERR_OUT_OF_MEMORY, "plan tables: hipHostMalloc failed");
  std::memcpy(dp->host, img.bytes.data(), total);
  e = hipMemcpyAsync(dp->dev, dp->host, total, hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) return hip_fail(e, "plan tables: hipMemcpyAsync");
  dp->bound.swap(bind);
  point_tables(dp.get(), static_cast<uint8_t*>(dp->dev), img);
  g_plans.push_front(dp);
  // Plans are keyed by shapes, so eviction happens only when more than
  // kMaxPlans list signatures alternate; hipFree waits for the device.
  while (g_plans.size() > kMaxPlans) g_plans.pop_back();
  *out = dp;
  return LM_OK;
}

// Record the end of this call's use of a plan (device scope: the event only
// orders later work on the same device).
lm_status release_plan(DevicePlan* dp, hipStream_t stream) {
  hipError_t e = hipSuccess;
  if (!dp->last_use) {
    e = hipEventCreateWithFlags(&dp->last_use, hipEventDisableTiming | hipEventDisableSystemFence);
    if (e != hipSuccess) return hip_fail(e, "plan: hipEventCreate");
  }
  e = hipEventRecord(dp->last_use, stream);
  if (e != hipSuccess) return hip_fail(e, "plan: hipEventRecord");
  dp->last_stream = stream;
  return LM_OK;
}

lm_status owned_workspace(size_t bytes, hipStream_t stream, OwnedWorkspace** out) {
  int device = 0;
  hipError_t e = hipGetDevice(&device);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  OwnedWorkspace* w = nullptr;
  for (auto& x : g_ws)
    if (x.device == device) w = &x;
  if (!w) {
    g_ws.emplace_back();
    w = &g_ws.back();
    w->device = device;
  }
  if (w->bytes < bytes) {
    if (w->ptr) (void)hipFree(w->ptr);   // waits for outstanding work on the device
    w->ptr = nullptr;
    w->bytes = 0;
    e = hipMalloc(&w->ptr, bytes);
    if (e != hipSuccess) return fail(LM_ERR_OUT_OF_MEMORY, "workspace: hipMalloc failed");
    w->bytes = bytes;
  }
  if (w->done && w->last != stream) {
    e = hipStreamWaitEvent(stream, w->done, 0);
    if (e != hipSuccess) return hip_fail(e, "workspace: hipStreamWaitEvent");
  }
  *out = w;
  return LM_OK;
}

// Record the end of this call's use of the owned workspace (device scope: the
// event only orders later work on the same device).
lm_status release_workspace(OwnedWorkspace* w, hipStream_t stream) {
  hipError_t e = hipSuccess;
  if (!w->done) {
    e = hipEventCreateWithFlags(&w->done, hipEventDisableTiming | hipEventDisableSystemFence);
    if (e != hipSuccess) return hip_fail(e, "workspace: hipEventCreate");
  }
  e = hipEventRecord(w->done, stream);
  if (e != hipSuccess) return hip_fail(e, "workspace: hipEventRecord");
  w->last = stream;
  return LM_OK;
}

// ---------------------------------------------------------------------------
// Launch sequence
// ---------------------------------------------------------------------------
struct Timer {
  hipStream_t stream;
  int phase;
  hipEvent_t start = nullptr, stop = nullptr;
  Timer(hipStream_t s, int ph) : stream(s), phase(ph) {
    if (!g_prof || g_prof_suppressed) return;
    if (get_event(&start) != hipSuccess || get_event(&stop) != hipSuccess ||
        hipEventRecord(start, stream) != hipSuccess) {
      start = stop = nullptr;
    }
  }
  void done() {
    if (!start) return;
    if (hipEventRecord(stop, stream) == hipSuccess) g_pending.push_back({phase, start, stop});
    start = nullptr;
  }
};

lm::StepConsts step_consts(double beta1, double beta2, double wd, double lr_muon,
                           double lr_lion, double eps, const lm_config* cfg, int64_t t) {
  lm::StepConsts k{};
  if (cfg) {   // AdamW: step count adam_step, or t + 1 (t counts from 0) when it is 0
    const double step = cfg->adam_step > 0 ? double(cfg->adam_step) : double(t) + 1.0;
    k.adam_lr = float(cfg->adam_lr);
    k.adam_b1 = float(cfg->adam_beta1);
    k.adam_omb1 = float(1.0 - cfg->adam_beta1);
    k.adam_b2 = float(cfg->adam_beta2);
    k.adam_omb2 = float(1.0 - cfg->adam_beta2);
    k.adam_eps = float(cfg->adam_eps);
    k.adam_wd = float(cfg->adam_wd);
    k.adam_c1 = float(1.0 / (1.0 - std::pow(cfg->adam_beta1, step)));
    k.adam_c2 = float(1.0 / (1.0 - std::pow(cfg->adam_beta2, step)));
  }
  k.beta1 = float(beta1);
  k.one_minus_beta1 = float(1.0 - beta1);
  k.beta2 = float(beta2);
  k.one_minus_beta2 = float(1.0 - beta2);
  k.lr_lion = float(lr_lion);
  k.lr_muon = float(lr_muon);
  k.wd = float(wd);
  k.eps = float(eps);
  return k;
}

// Optional per-input-tensor outputs of the adaptive step (device pointers).
struct AdaptiveOut {
  int32_t* decisions = nullptr;
  double* srank = nullptr;
};

lm_status enqueue(const DevicePlan& dp, const lm::StepConsts& k, const lm_config& cfg, void* ws,
                  bool store_o, const AdaptiveOut& aout, hipStream_t stream) {
  const Plan& p = dp.plan;
  hipError_t e = hipSuccess;
  uint8_t* wsb = static_cast<uint8_t*>(ws);
  int32_t* decide = nullptr;
  if (p.adaptive && !p.mats.empty()) {
    // Appendix G: stable rank of each candidate's momentum, before this
    // step updates it, and the per-matrix decision, all on the device.
    decide = reinterpret_cast<int32_t*>(wsb + p.ws_decide_off);
    lm::SrankLaunch sl;
    sl.mats = dp.d_mats;
    sl.bind = dp.d_bind;
    sl.tab = dp.d_sr_tab;
    sl.rd_start = dp.d_rd_start;
    sl.tensor_mat = dp.d_tensor_mat;
    sl.n_mats = int32_t(p.mats.size());
    sl.n_chunks = p.rd_start.back();
    sl.n_inputs = int32_t(p.tensor_mat.size());
    sl.ws = ws;
    sl.decide = decide;
    sl.decisions_out = aout.decisions;
    sl.srank_out = aout.srank;
    sl.alpha = cfg.adaptive_alpha;
    Timer t(stream, LM_PHASE_SRANK);
    const int steps = cfg.adaptive_power_steps;
    // Every pass reads all candidate momenta; odd passes walk them in
    // reverse (classes and blocks), so a pass starts with the data the
    // previous one read last, which the last-level cache still holds.
    const size_t nc = p.sr_classes.size();
    for (int i = 0; i <= steps && e == hipSuccess; ++i) {
      const bool rev = (i & 1) != 0;
      for (size_t j = 0; j < nc; ++j) {
        const Plan::SrClass& c = p.sr_classes[rev ? nc - 1 - j : j];
        e = lm::launch_srank_pass(sl, c.kind, c.bucket, c.first, c.count, i == 0, i == steps,
                                  rev, stream);
        if (e != hipSuccess) break;
      }
      if (e == hipSuccess && i < steps) e = lm::launch_srank_reduce(sl, stream);
    }
    if (e == hipSuccess) e = lm::launch_srank_decide(sl, stream);
    t.done();
    if (e != hipSuccess) return hip_fail(e, "stable-rank kernel launch");
  } else if (p.adaptive && (aout.decisions || aout.srank)) {
    // no candidate matrix: every output entry says "not a candidate"
    lm::SrankLaunch sl{};
    sl.tensor_mat = dp.d_tensor_mat;
    sl.n_inputs = int32_t(p.tensor_mat.size());
    sl.decisions_out = aout.decisions;
    sl.srank_out = aout.srank;
    e = lm::launch_srank_decide(sl, stream);
    if (e != hipSuccess) return hip_fail(e, "stable-rank kernel launch");
  }
  if (!p.lion.empty()) {
    lm::LionLaunch l;
    l.tensors = dp.d_lion;
    l.bind = dp.d_bind;
    l.block_start = dp.d_lion_start;
    l.n_tensors = int32_t(p.lion.size());
    l.n_blocks = p.lion_block_start.back();
    l.decide = decide;
    l.k = k;
    Timer t(stream, LM_PHASE_LION);
    e = lm::launch_lion(l, stream);
    t.done();
    if (e != hipSuccess) return hip_fail(e, "lion kernel launch");
  }
  if (p.mats.empty()) return LM_OK;
  float* partials = reinterpret_cast<float*>(wsb + p.ws_partials_off);
  float* rscale = reinterpret_cast<float*>(wsb + p.ws_rscale_off);
  lm::PrepLaunch pl;
  pl.mats = dp.d_mats;
  pl.bind = dp.d_bind;
  pl.prep_start = dp.d_prep_start;
  pl.n_mats = int32_t(p.mats.size());
  pl.n_tiles = p.prep_start.back();
  pl.ws = ws;
  pl.partials = partials;
  pl.rscale = rscale;
  pl.decide = decide;
  pl.k = k;
  {
    Timer t(stream, LM_PHASE_PREP);
    e = lm::launch_prep(pl, stream);
    t.done();
    if (e != hipSuccess) return hip_fail(e, "prep kernel launch");
  }
  {
    Timer t(stream, LM_PHASE_NORM);
    e = lm::launch_norm(pl, stream);
    t.done();
    if (e != hipSuccess) return hip_fail(e, "norm kernel launch");
  }
  lm::GemmLaunch gl;
  gl.mats = dp.d_mats;
  gl.bind = dp.d_bind;
  gl.chip = p.chip;
  gl.ws = ws;
  gl.rscale = rscale;
  gl.store_o = store_o ? 1 : 0;
  gl.lr = k.lr_muon;
  gl.wd = k.wd;
  gl.decide = decide;
  const lm::GemmMode modes[3] = {lm::kGram, lm::kPoly, lm::kApply};
  const int phases[3] = {LM_PHASE_GRAM, LM_PHASE_POLY, LM_PHASE_APPLY};
  for (int it = 0; it < cfg.ns_steps; ++it) {
    const bool sched = cfg.ns_schedule_steps != 0;
    gl.a = float(sched ? cfg.ns_schedule[it][0] : cfg.ns_a);
    gl.b = float(sched ? cfg.ns_schedule[it][1] : cfg.ns_b);
    gl.c = float(sched ? cfg.ns_schedule[it][2] : cfg.ns_c);
    gl.src = it & 1;
    gl.first = it == 0;
    gl.last = it == cfg.ns_steps - 1;
    for (int st3 = 0; st3 < 3; ++st3) {
      Timer t(stream, phases[st3]);
      for (int pr = 0; pr < 2; ++pr) {   // bf16 matrices, then fp32 matrices
        const lm::XcdSplit& sp = st3 == 0 ? p.gram_split[pr] : (st3 == 1 ? p.poly_split[pr]
                                                                          : p.apply_split[pr]);
        if (sp.max_count == 0) continue;
        gl.tasks = dp.d_tasks[pr][st3];
        gl.split = dp.d_splits + pr * 4 + st3;
        gl.max_count = sp.max_count;
        gl.fp32 = pr;
        gl.tile = p.tile[pr][st3];
        // the apply's last round as smaller tiles, in the same launch
        const bool tail = st3 == 2 && p.apply_tail_split[pr].max_count > 0;
        gl.tail_tasks = tail ? dp.d_tasks[pr][3] : nullptr;
        gl.tail_split = tail ? dp.d_splits + pr * 4 + 3 : nullptr;
        gl.tail_max_count = tail ? p.apply_tail_split[pr].max_count : 0;
        gl.tail_tile = tail ? p.tail_tile[pr] : 0;
        e = lm::launch_gemm(modes[st3], gl, stream);
        if (e != hipSuccess) return hip_fail(e, "Newton-Schulz kernel launch");
      }
      t.done();
    }
  }
  return LM_OK;
}

lm_status check_config(const lm_config* cfg) {
  if (cfg->struct_size != sizeof(lm_config)) return fail(LM_ERR_INVALID_ARGUMENT, "lm_config.struct_size mismatch");
  if (cfg->ns_steps < 1 || cfg->ns_steps > 64) return fail(LM_ERR_INVALID_ARGUMENT, "ns_steps must lie in [1, 64]");
  if (!std::isfinite(cfg->ns_a) || !std::isfinite(cfg->ns_b) || !std::isfinite(cfg->ns_c))
    return fail(LM_ERR_INVALID_ARGUMENT, "Newton-Schulz coefficients must be finite");
  if (!(cfg->ns_eps >= 0.0f) || !std::isfinite(cfg->ns_eps)) return fail(LM_ERR_INVALID_ARGUMENT, "ns_eps must be finite and >= 0");
  if (cfg->ns_precision != LM_NS_BF16 && cfg->ns_precision != LM_NS_FP32)
    return fail(LM_ERR_INVALID_ARGUMENT, "unknown ns_precision");
  if (cfg->ns_scale_mode != LM_NS_SCALE_NONE && cfg->ns_scale_mode != LM_NS_SCALE_RMS02)
    return fail(LM_ERR_INVALID_ARGUMENT, "unknown ns_scale_mode");
  if (cfg->ns_bf16_min_side < 0) return fail(LM_ERR_INVALID_ARGUMENT, "ns_bf16_min_side must be >= 0");
  if (cfg->reserved != 0 || cfg->reserved2 != 0)
    return fail(LM_ERR_INVALID_ARGUMENT, "lm_config reserved fields must be 0");
  if (!(cfg->adam_beta1 >= 0.0 && cfg->adam_beta1 < 1.0) ||
      !(cfg->adam_beta2 >= 0.0 && cfg->adam_beta2 < 1.0))
    return fail(LM_ERR_INVALID_ARGUMENT, "adam betas must lie in [0, 1)");
  if (!(cfg->adam_lr >= 0.0) || !std::isfinite(cfg->adam_lr) || !(cfg->adam_eps >= 0.0) ||
      !std::isfinite(cfg->adam_eps) || !(cfg->adam_wd >= 0.0) || !std::isfinite(cfg->adam_wd))
    return fail(LM_ERR_INVALID_ARGUMENT, "adam_lr, adam_eps and adam_wd must be finite and >= 0");
  if (!(cfg->adaptive_alpha >= 0.0 && cfg->adaptive_alpha <= 1.0))
    return fail(LM_ERR_INVALID_ARGUMENT, "adaptive_alpha must be 0 (off) or lie in (0, 1]");
  if (cfg->adaptive_power_steps < 0 || cfg->adaptive_power_steps > 64)
    return fail(LM_ERR_INVALID_ARGUMENT, "adaptive_power_steps must lie in [0, 64]");
  if (cfg->reserved3 != 0) return fail(LM_ERR_INVALID_ARGUMENT, "lm_config reserved fields must be 0");
  if (cfg->adam_step < 0) return fail(LM_ERR_INVALID_ARGUMENT, "adam_step must be >= 0 (0: t + 1)");
  if (cfg->ns_schedule_steps != 0) {
    if (cfg->ns_schedule_steps != cfg->ns_steps || cfg->ns_steps > LM_MAX_NS_SCHEDULE)
      return fail(LM_ERR_INVALID_ARGUMENT,
                  "ns_schedule_steps must be 0 or equal ns_steps (at most 16)");
    for (int k = 0; k < cfg->ns_steps; ++k)
      for (int j = 0; j < 3; ++j)
        if (!std::isfinite(cfg->ns_schedule[k][j]))
          return fail(LM_ERR_INVALID_ARGUMENT, "ns_schedule coefficients must be finite");
  }
  return LM_OK;
}

lm::StepKind step_kind(const lm_config& cfg, int64_t t, int32_t P) {
  if (cfg.adaptive_alpha > 0.0) return lm::StepKind::kAdaptive;
  return lm::is_muon_step(t, P) ? lm::StepKind::kMuon : lm::StepKind::kLion;
}

lm::NsPrecision precision_of(const lm_config& cfg) {
  lm::NsPrecision p;
  p.all_fp32 = cfg.ns_precision == LM_NS_FP32;
  p.bf16_min_side = cfg.ns_bf16_min_side;
  return p;
}

std::vector<TensorIn> gather(float* const* params, const float* const* grads, float* const* momentum,
                             float* const* second_moment, const lm_shape* shapes, int32_t n) {
  std::vector<TensorIn> v(size_t(n > 0 ? n : 0));
  for (int32_t i = 0; i < n; ++i) {
    v[i].w = params[i];
    v[i].g = grads[i];
    v[i].m = momentum[i];
    v[i].v = (second_moment && (shapes[i].flags & lm::kFlagAdamW)) ? second_moment[i] : nullptr;
    v[i].rows = shapes[i].rows;
    v[i].cols = shapes[i].cols;
    v[i].flags = shapes[i].flags;
    v[i].reserved = shapes[i].reserved;
  }
  return v;
}

lm_status step_impl(float* const* params, const float* const* grads, float* const* momentum,
                    float* const* second_moment, const lm_shape* shapes, int32_t n, int64_t t,
                    int32_t P, double beta1,
                    double beta2, double wd, const lm_config* cfg, void* workspace,
                    size_t workspace_bytes, const AdaptiveOut& aout, hipStream_t stream) {
  if (cfg == nullptr) return fail(LM_ERR_INVALID_ARGUMENT, "null config");
  lm_status cs = check_config(cfg);
  if (cs != LM_OK) return cs;
  std::string err;
  Status st = lm::validate_scalars(t, P, beta1, beta2, wd, cfg->lr_muon, cfg->lr_lion, &err);
  if (st != Status::kOk) return fail(to_c(st), err);
  if (n < 0) return fail(LM_ERR_INVALID_ARGUMENT, "n_tensors must be >= 0");
  if (n == 0) return LM_OK;
  if (!params || !grads || !momentum || !shapes) return fail(LM_ERR_INVALID_ARGUMENT, "null tensor array");
  if ((workspace == nullptr) != (workspace_bytes == 0))
    return fail(LM_ERR_INVALID_ARGUMENT, "workspace and workspace_bytes must both be set or both be 0");
  if (workspace && (reinterpret_cast<uintptr_t>(workspace) & 255u))
    return fail(LM_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  std::vector<TensorIn> x = gather(params, grads, momentum, second_moment, shapes, n);
  st = lm::validate_tensors(x.data(), n, &err);
  if (st != Status::kOk) return fail(to_c(st), err);
  bool any = false;
  for (const TensorIn& ti : x) any = any || (ti.rows > 0 && ti.cols > 0);
  const lm::StepKind kind = step_kind(*cfg, t, P);
  if (!any && !(kind == lm::StepKind::kAdaptive && (aout.decisions || aout.srank)))
    return LM_OK;                                  // only empty tensors: nothing to do
  const bool rms02 = cfg->ns_scale_mode == LM_NS_SCALE_RMS02;

  std::lock_guard<std::mutex> lock(g_mu);
  std::shared_ptr<DevicePlan> dp;
  lm_status s = get_plan(x.data(), n, kind, precision_of(*cfg), rms02, stream, &dp);
  if (s != LM_OK) return s;
  void* ws = workspace;
  OwnedWorkspace* ow = nullptr;
  if (dp->plan.ws_bytes > 0) {
    if (workspace) {
      if (workspace_bytes < dp->plan.ws_bytes)
        return fail(LM_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than lionmuon_workspace_bytes");
    } else {
      s = owned_workspace(dp->plan.ws_bytes, stream, &ow);
      if (s != LM_OK) return s;
      ws = ow->ptr;
    }
  }
  s = enqueue(*dp, step_consts(beta1, beta2, wd, cfg->lr_muon, cfg->lr_lion, cfg->ns_eps, cfg, t),
              *cfg, ws, false, aout, stream);
  {                                      // also after a partial enqueue
    const lm_status r = release_plan(dp.get(), stream);
    if (s == LM_OK) s = r;
  }
  if (ow) {
    const lm_status r = release_workspace(ow, stream);
    if (s == LM_OK) s = r;
  }
  return s;
}

// ---------------------------------------------------------------------------
// No-allocation entry point
// ---------------------------------------------------------------------------
// Per device: the scratch array's device address and which list signature's
// tables and which addresses it holds. Calls on one device share the array
// and must not overlap.
struct StaticScratch {
  int device = -1;
  uint8_t* ptr = nullptr;
  std::vector<uint8_t> key;               // signature whose tables are resident
  DevicePlan view;                        // the plan, its tables in scratch (not owned)
  size_t ws_off = 0;                      // workspace offset in scratch
};
std::vector<std::unique_ptr<StaticScratch>> g_static;

lm_status step_noalloc_impl(float* const* params, const float* const* grads,
                            float* const* momentum, float* const* second_moment,
                            const lm_shape* shapes, int32_t n, int64_t t, int32_t P, double beta1,
                            double beta2, double wd, const lm_config* cfg, hipStream_t stream) {
  if (cfg == nullptr) return fail(LM_ERR_INVALID_ARGUMENT, "null config");
  lm_status cs = check_config(cfg);
  if (cs != LM_OK) return cs;
  std::string err;
  Status st = lm::validate_scalars(t, P, beta1, beta2, wd, cfg->lr_muon, cfg->lr_lion, &err);
  if (st != Status::kOk) return fail(to_c(st), err);
  if (n < 0) return fail(LM_ERR_INVALID_ARGUMENT, "n_tensors must be >= 0");
  if (n == 0) return LM_OK;
  if (!params || !grads || !momentum || !shapes) return fail(LM_ERR_INVALID_ARGUMENT, "null tensor array");
  std::vector<TensorIn> x = gather(params, grads, momentum, second_moment, shapes, n);
  st = lm::validate_tensors(x.data(), n, &err);
  if (st != Status::kOk) return fail(to_c(st), err);
  bool any = false;
  for (const TensorIn& ti : x) any = any || (ti.rows > 0 && ti.cols > 0);
  if (!any) return LM_OK;
  const lm::StepKind kind = step_kind(*cfg, t, P);
  const bool rms02 = cfg->ns_scale_mode == LM_NS_SCALE_RMS02;
  const lm::NsPrecision prec = precision_of(*cfg);

  std::lock_guard<std::mutex> lock(g_mu);
  int device = 0;
  hipError_t e = hipGetDevice(&device);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  StaticScratch* sc = nullptr;
  for (auto& d : g_static)
    if (d->device == device) sc = d.get();
  if (!sc) {
    void* ptr = nullptr;
    e = lm::scratch_address(device, &ptr);
    if (e != hipSuccess) return hip_fail(e, "scratch: hipGetSymbolAddress");
    g_static.push_back(std::make_unique<StaticScratch>());
    sc = g_static.back().get();
    sc->device = device;
    sc->ptr = static_cast<uint8_t*>(ptr);
  }
  std::vector<uint8_t> key = plan_key(device, x.data(), n, kind, prec, rms02);
  std::vector<lm::TensorPtrs> bind = binding_of(x.data(), n);
  if (key != sc->key) {
    // new signature: plan on the host, check the size limit, then upload
    // the tables (and the binding) into the scratch array
    Plan p;
    st = lm::build_plan(x.data(), n, kind, prec, rms02, chip_of(device), &p, &err);
    if (st != Status::kOk) return fail(to_c(st), err);
    TableImage img;
    pack_tables(p, bind, &img);
    const size_t ws_off = align256(img.bytes.size());
    const size_t need = ws_off + p.ws_bytes;
    if (need > lm::kScratchBytes)
      return fail(LM_ERR_UNSUPPORTED,
                  "lionmuon_step_noalloc: this list needs " + std::to_string(need) +
                      " bytes of device scratch (plan tables and workspace); its static scratch "
                      "holds at most " + std::to_string(lm::kScratchBytes) +
                      " bytes (use lionmuon_step_ex for larger lists)");
    sc->key.clear();                       // invalid until the upload is enqueued
    e = lm::launch_upload(sc->ptr, img.bytes.data(), img.bytes.size(), stream);
    if (e != hipSuccess) return hip_fail(e, "scratch: table upload");
    sc->view.plan = std::move(p);
    sc->view.bound.swap(bind);
    point_tables(&sc->view, sc->ptr, img);
    sc->ws_off = ws_off;
    sc->key.swap(key);
  } else if (!same_binding(sc->view.bound, bind)) {
    e = lm::launch_upload(sc->view.d_bind, bind.data(), bind.size() * sizeof(lm::TensorPtrs),
                          stream);
    if (e != hipSuccess) return hip_fail(e, "scratch: address table upload");
    sc->view.bound.swap(bind);
  }
  void* ws = sc->view.plan.ws_bytes > 0 ? sc->ptr + sc->ws_off : nullptr;
  g_prof_suppressed = true;
  const lm_status s = enqueue(sc->view, step_consts(beta1, beta2, wd, cfg->lr_muon, cfg->lr_lion,
                                                    cfg->ns_eps, cfg, t),
                              *cfg, ws, false, AdaptiveOut(), stream);
  g_prof_suppressed = false;
  return s;
}

}  // namespace

extern "C" {

void lionmuon_config_default(lm_config* cfg) {
  if (!cfg) return;
  std::memset(cfg, 0, sizeof(*cfg));
  cfg->struct_size = sizeof(lm_config);
  cfg->ns_steps = 5;
  cfg->ns_a = 3.4445;
  cfg->ns_b = -4.7750;
  cfg->ns_c = 2.0315;
  cfg->ns_eps = 1e-7;
  cfg->ns_precision = LM_NS_BF16;
  cfg->ns_scale_mode = LM_NS_SCALE_NONE;
  cfg->lr_muon = 0.0;
  cfg->lr_lion = 0.0;
  cfg->ns_bf16_min_side = 64;
  cfg->reserved = 0;
  cfg->ns_schedule_steps = 0;
  cfg->reserved2 = 0;
  cfg->adam_lr = 1e-3;
  cfg->adam_beta1 = 0.8;
  cfg->adam_beta2 = 0.999;
  cfg->adam_eps = 1e-8;
  cfg->adam_wd = 0.0;
  cfg->adaptive_alpha = 0.0;
  cfg->adaptive_power_steps = 5;
  cfg->reserved3 = 0;
  cfg->adam_step = 0;
}

lm_status lionmuon_step(float* const* params, const float* const* grads, float* const* momentum,
                        const lm_shape* shapes, int32_t n_tensors, int64_t t, int32_t P,
                        double beta1, double beta2, double lr, double wd, hipStream_t stream) {
  lm_config cfg;
  lionmuon_config_default(&cfg);
  cfg.lr_muon = lr;
  cfg.lr_lion = lr;
  return step_impl(params, grads, momentum, nullptr, shapes, n_tensors, t, P, beta1, beta2, wd,
                   &cfg, nullptr, 0, AdaptiveOut(), stream);
}

lm_status lionmuon_step_ex(float* const* params, const float* const* grads, float* const* momentum,
                           float* const* second_moment, const lm_shape* shapes, int32_t n_tensors,
                           int64_t t, int32_t P, double beta1, double beta2, double wd,
                           const lm_config* cfg, void* workspace, size_t workspace_bytes,
                           hipStream_t stream) {
  return step_impl(params, grads, momentum, second_moment, shapes, n_tensors, t, P, beta1, beta2,
                   wd, cfg, workspace, workspace_bytes, AdaptiveOut(), stream);
}

lm_status lionmuon_step_noalloc(float* const* params, const float* const* grads,
                                float* const* momentum, float* const* second_moment,
                                const lm_shape* shapes, int32_t n_tensors, int64_t t, int32_t P,
                                double beta1, double beta2, double wd, const lm_config* cfg,
                                hipStream_t stream) {
  return step_noalloc_impl(params, grads, momentum, second_moment, shapes, n_tensors, t, P, beta1,
                           beta2, wd, cfg, stream);
}

lm_status lionmuon_step_adaptive(float* const* params, const float* const* grads,
                                 float* const* momentum, float* const* second_moment,
                                 const lm_shape* shapes, int32_t n_tensors, int64_t t, double beta1,
                                 double beta2, double wd, const lm_config* cfg, void* workspace,
                                 size_t workspace_bytes, int32_t* decisions, double* stable_rank,
                                 hipStream_t stream) {
  if (cfg == nullptr) return fail(LM_ERR_INVALID_ARGUMENT, "null config");
  if (!(cfg->adaptive_alpha > 0.0))
    return fail(LM_ERR_INVALID_ARGUMENT, "lionmuon_step_adaptive needs adaptive_alpha in (0, 1]");
  if (n_tensors > 0) {
    const uintptr_t d = reinterpret_cast<uintptr_t>(decisions);
    const uintptr_t r = reinterpret_cast<uintptr_t>(stable_rank);
    if ((d & 3u) || (r & 7u))
      return fail(LM_ERR_INVALID_ARGUMENT, "decisions / stable_rank must be int32 / fp64 aligned");
    if (d && r && d < r + uintptr_t(n_tensors) * 8u && r < d + uintptr_t(n_tensors) * 4u)
      return fail(LM_ERR_INVALID_ARGUMENT, "decisions and stable_rank overlap");
  }
  AdaptiveOut aout;
  aout.decisions = n_tensors > 0 ? decisions : nullptr;
  aout.srank = n_tensors > 0 ? stable_rank : nullptr;
  return step_impl(params, grads, momentum, second_moment, shapes, n_tensors, t, 0, beta1, beta2,
                   wd, cfg, workspace, workspace_bytes, aout, stream);
}

lm_status lionmuon_workspace_bytes(const lm_shape* shapes, int32_t n_tensors, const lm_config* cfg,
                                   size_t* out_bytes) {
  lm_plan_info info;
  lm_status s = lionmuon_plan_info(shapes, n_tensors, 0, 1, cfg, &info);
  if (s != LM_OK) return s;
  if (!out_bytes) return fail(LM_ERR_INVALID_ARGUMENT, "null out_bytes");
  *out_bytes = info.workspace_bytes;
  return LM_OK;
}

lm_status lionmuon_plan_info(const lm_shape* shapes, int32_t n, int64_t t, int32_t P,
                             const lm_config* cfg, lm_plan_info* out) {
  if (!out) return fail(LM_ERR_INVALID_ARGUMENT, "null output");
  lm_config def;
  lionmuon_config_default(&def);
  if (!cfg) cfg = &def;
  lm_status cs = check_config(cfg);
  if (cs != LM_OK) return cs;
  if (n < 0) return fail(LM_ERR_INVALID_ARGUMENT, "n_tensors must be >= 0");
  if (n > 0 && !shapes) return fail(LM_ERR_INVALID_ARGUMENT, "null shapes");
  if (t < 0 || P < 0) return fail(LM_ERR_INVALID_ARGUMENT, "t and P must be >= 0");
  // Synthetic, distinct, 16-byte aligned addresses: only shapes matter here.
  std::vector<TensorIn> x(static_cast<size_t>(n));
  uintptr_t addr = 4096;
  for (int32_t i = 0; i < n; ++i) {
    x[i].rows = shapes[i].rows;
    x[i].cols = shapes[i].cols;
    x[i].flags = shapes[i].flags;
    x[i].reserved = shapes[i].reserved;
    if (x[i].rows < 0 || x[i].cols < 0) continue;    // rejected by validate_tensors
    const uintptr_t bytes = (uintptr_t(x[i].rows) * uintptr_t(x[i].cols) * 4u + 15u) & ~uintptr_t(15);
    x[i].w = reinterpret_cast<float*>(addr); addr += bytes + 16;
    x[i].g = reinterpret_cast<const float*>(addr); addr += bytes + 16;
    x[i].m = reinterpret_cast<float*>(addr); addr += bytes + 16;
    x[i].v = reinterpret_cast<float*>(addr); addr += bytes + 16;
  }
  std::string err;
  Status st = lm::validate_tensors(x.data(), n, &err);
  if (st != Status::kOk) return fail(to_c(st), err);
  Plan p;
  st = lm::build_plan(x.data(), n, step_kind(*cfg, t, P), precision_of(*cfg),
                      cfg->ns_scale_mode == LM_NS_SCALE_RMS02, current_chip(), &p, &err);
  if (st != Status::kOk) return fail(to_c(st), err);
  std::memset(out, 0, sizeof(*out));
  out->n_tensors = p.n_tensors;
  out->n_lion = int32_t(p.lion.size()) - p.n_adamw - (p.adaptive ? int32_t(p.mats.size()) : 0);
  out->n_adamw = p.n_adamw;
  out->adamw_elements = p.adamw_elements;
  out->n_muon = int32_t(p.mats.size());
  out->n_shape_classes = p.n_shape_classes;
  out->lion_elements = p.lion_elements;
  out->muon_elements = p.muon_elements;
  out->gram_tiles = int64_t(p.gram[0].size() + p.gram[1].size());
  out->poly_tiles = int64_t(p.poly[0].size() + p.poly[1].size());
  out->apply_tiles = int64_t(p.apply[0].size() + p.apply[1].size() + p.apply_tail[0].size() +
                             p.apply_tail[1].size());
  out->ns_flops = lm::ns_flops_symmetric(p, cfg->ns_steps);
  out->ns_flops_dense = lm::ns_flops_dense(p, cfg->ns_steps);
  out->lion_bytes = 20.0 * double(p.lion_elements) + 28.0 * double(p.adamw_elements);
  out->workspace_bytes = p.ws_bytes;
  if (p.adaptive) {
    // M read once per pass (power steps + 1), plus the fp64 partial products
    // written and read back once per power step
    double part = 0.0;
    for (const lm::MuonMat& mm : p.mats) part += 16.0 * double(mm.sr_blocks) * double(mm.s);
    out->srank_bytes = 4.0 * double(p.candidate_elements) * (cfg->adaptive_power_steps + 1) +
                       part * cfg->adaptive_power_steps;
  }
  return LM_OK;
}

lm_status lionmuon_ns(const float* X, float* O, int64_t rows, int64_t cols, int32_t batch,
                      const lm_config* cfg, void* workspace, size_t workspace_bytes,
                      hipStream_t stream) {
  lm_config def;
  lionmuon_config_default(&def);
  if (!cfg) cfg = &def;
  lm_status cs = check_config(cfg);
  if (cs != LM_OK) return cs;
  if (batch < 0 || rows < 0 || cols < 0) return fail(LM_ERR_INVALID_ARGUMENT, "negative size");
  if (batch == 0 || rows == 0 || cols == 0) return LM_OK;
  if (!X || !O) return fail(LM_ERR_INVALID_ARGUMENT, "null X or O");
  if (rows < 2 || cols < 2) return fail(LM_ERR_UNSUPPORTED, "Newton-Schulz hook needs rows, cols >= 2");
  if ((workspace == nullptr) != (workspace_bytes == 0))
    return fail(LM_ERR_INVALID_ARGUMENT, "workspace and workspace_bytes must both be set or both be 0");
  if (workspace && (reinterpret_cast<uintptr_t>(workspace) & 255u))
    return fail(LM_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
  const int64_t numel = rows * cols;
  const uintptr_t xb = reinterpret_cast<uintptr_t>(X), ob = reinterpret_cast<uintptr_t>(O);
  const uintptr_t bytes = uintptr_t(numel) * uintptr_t(batch) * 4u;
  if (xb < ob + bytes && ob < xb + bytes) return fail(LM_ERR_INVALID_ARGUMENT, "X and O overlap");
  if ((xb | ob) & 3u) return fail(LM_ERR_INVALID_ARGUMENT, "X and O must be 4-byte aligned");
  // Each matrix is a Muon tensor with G = X, no momentum (beta1 = 0) and an
  // output epilogue that stores kappa * NS_K(X) into O.
  std::vector<TensorIn> x(static_cast<size_t>(batch));
  for (int32_t b = 0; b < batch; ++b) {
    x[b].w = O + b * numel;
    x[b].g = X + b * numel;
    x[b].m = nullptr;
    x[b].v = nullptr;
    x[b].rows = rows;
    x[b].cols = cols;
    x[b].flags = 0;
    x[b].reserved = 0;
  }
  const bool rms02 = cfg->ns_scale_mode == LM_NS_SCALE_RMS02;
  std::lock_guard<std::mutex> lock(g_mu);
  std::shared_ptr<DevicePlan> dp;
  lm_status s = get_plan(x.data(), batch, lm::StepKind::kMuon, precision_of(*cfg), rms02, stream,
                         &dp);
  if (s != LM_OK) return s;
  void* ws = workspace;
  OwnedWorkspace* ow = nullptr;
  if (workspace) {
    if (workspace_bytes < dp->plan.ws_bytes)
      return fail(LM_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than lionmuon_workspace_bytes");
  } else {
    s = owned_workspace(dp->plan.ws_bytes, stream, &ow);
    if (s != LM_OK) return s;
    ws = ow->ptr;
  }
  s = enqueue(*dp, step_consts(0.0, 0.0, 0.0, 0.0, 0.0, cfg->ns_eps, nullptr, 0), *cfg, ws, true,
              AdaptiveOut(), stream);
  {
    const lm_status r = release_plan(dp.get(), stream);
    if (s == LM_OK) s = r;
  }
  if (ow) {
    const lm_status r = release_workspace(ow, stream);
    if (s == LM_OK) s = r;
  }
  return s;
}

lm_status lionmuon_profiling_enable(int32_t enable) {
  std::lock_guard<std::mutex> lock(g_mu);
  g_prof = enable != 0;
  return LM_OK;
}

lm_status lionmuon_profiling_read(lm_phase_times* out) {
  if (!out) return fail(LM_ERR_INVALID_ARGUMENT, "null output");
  std::lock_guard<std::mutex> lock(g_mu);
  for (const PendingEvent& pe : g_pending) {
    hipError_t e = hipEventSynchronize(pe.stop);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    float ms = 0.0f;
    e = hipEventElapsedTime(&ms, pe.start, pe.stop);
    if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
    g_times.ms[pe.phase] += ms;
    g_times.launches[pe.phase] += 1;
    g_event_pool.push_back(pe.start);
    g_event_pool.push_back(pe.stop);
  }
  g_pending.clear();
  *out = g_times;
  return LM_OK;
}

lm_status lionmuon_profiling_reset(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  for (const PendingEvent& pe : g_pending) {
    (void)hipEventSynchronize(pe.stop);
    g_event_pool.push_back(pe.start);
    g_event_pool.push_back(pe.stop);
  }
  g_pending.clear();
  std::memset(&g_times, 0, sizeof(g_times));
  return LM_OK;
}

void lionmuon_release(void) {
  std::lock_guard<std::mutex> lock(g_mu);
  g_plans.clear();
  for (auto& reg : g_ring.inflight) {
    (void)hipEventSynchronize(reg.done);
    g_ring.pool.push_back(reg.done);
  }
  g_ring.inflight.clear();
  for (hipEvent_t e : g_ring.pool) (void)hipEventDestroy(e);
  g_ring.pool.clear();
  if (g_ring.host) (void)hipHostFree(g_ring.host);
  g_ring.host = nullptr;
  g_ring.cap = 0;
  for (auto& w : g_ws) {
    if (w.ptr) (void)hipFree(w.ptr);
    if (w.done) (void)hipEventDestroy(w.done);
  }
  g_ws.clear();
  for (const PendingEvent& pe : g_pending) {
    (void)hipEventSynchronize(pe.stop);
    g_event_pool.push_back(pe.start);
    g_event_pool.push_back(pe.stop);
  }
  g_pending.clear();
  for (hipEvent_t e : g_event_pool) (void)hipEventDestroy(e);
  g_event_pool.clear();
}

const char* lionmuon_status_string(lm_status s) {
  switch (s) {
    case LM_OK: return "LM_OK";
    case LM_ERR_INVALID_ARGUMENT: return "LM_ERR_INVALID_ARGUMENT";
    case LM_ERR_UNSUPPORTED: return "LM_ERR_UNSUPPORTED";
    case LM_ERR_OUT_OF_MEMORY: return "LM_ERR_OUT_OF_MEMORY";
    case LM_ERR_WORKSPACE_TOO_SMALL: return "LM_ERR_WORKSPACE_TOO_SMALL";
    case LM_ERR_HIP: return "LM_ERR_HIP";
  }
  return "unknown lm_status";
}

const char* lionmuon_last_error(void) { return g_last_error.c_str(); }

int32_t lionmuon_abi_version(void) { return LIONMUON_ABI_VERSION; }

}  // extern "C"
