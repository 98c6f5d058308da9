// Launch-side runtime: per-device plan images, family dispatch and the
// watchdog status word.
#include <hip/hip_runtime.h>

#include <cstring>
#include <string>
#include <utility>
#include <vector>

#include "bfs_internal.h"

// The fixed device array of bfs_run_noalloc (see below).  Host code never
// names it except in the one hipGetSymbolAddress call.
static __device__ __align__(256) unsigned char scratch[BFS_NOALLOC_MAX_IMAGE_BYTES];

namespace bfs {

namespace {

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace

std::vector<DevWait> device_waits(const bfs_plan *p) {
  std::vector<DevWait> w(p->formulas.size());
  for (size_t d = 0; d < w.size(); ++d) {
    const bfs_formula &f = p->formulas[d];
    DevWait x{};
    x.dep = (int32_t)d;
    if (p->mode == BFS_MODE_BARRIER) {
      const bfs_static_wait &s = p->static_waits[d];
      x.counter = s.prd_engine;
      x.prd_engine = s.prd_engine;
      x.ordinal = s.ordinal;
      x.active = s.same_region;
    } else {
      x.counter = f.counter;
      x.prd_engine = f.prd_engine;
      x.loop_S = f.loop_S;
      x.loop_P = f.loop_P;
      x.k = f.k;
      x.expr_sub = f.expr_sub;
      x.N = f.N;
      x.K = f.K;
      x.needs_mask = f.needs_mask;
      x.active = f.kase != 4;
      x.snap_slots = f.snap_slots;
      x.snap_off = p->snap_off.empty() ? 0 : p->snap_off[d];
      x.linear = f.kase == 6 ? 1 : 0;
    }
    w[d] = x;
  }
  return w;
}

namespace {

// Table order in a packed plan image.
enum { T_CODE, T_COFF, T_WAIT, T_OP, T_ARGS, T_IW, T_WL, T_UPD, T_LP, T_N };
// The first kErrBytes of an image hold the error words (zero at upload).
constexpr size_t kErrBytes = 256;

// Packs the plan's device tables into plan->packed once (caller holds
// plan->dev_mu).
void pack_tables(bfs_plan *plan) {
  if (!plan->packed.empty()) return;
  const std::vector<DevWait> waits = device_waits(plan);
  const std::pair<const void *, size_t> src[T_N] = {
      {plan->code.data(), plan->code.size() * 4},
      {plan->code_off.data(), plan->code_off.size() * 4},
      {waits.data(), waits.size() * sizeof(DevWait)},
      {plan->instr_opcode.data(), plan->instr_opcode.size() * 4},
      {plan->instr_args.data(), plan->instr_args.size() * 4},
      {plan->instr_wait_off.data(), plan->instr_wait_off.size() * 4},
      {plan->instr_wait_list.data(), plan->instr_wait_list.size() * 4},
      {plan->instr_update.data(), plan->instr_update.size() * 4},
      {plan->loop_parent.data(), plan->loop_parent.size() * 4}};
  plan->packed_off.assign(T_N, 0);
  size_t off = kErrBytes;
  for (int t = 0; t < T_N; ++t) {
    off = align_up(off, 256);
    plan->packed_off[t] = off;
    off += src[t].second > 0 ? src[t].second : 4;
  }
  plan->packed.assign(align_up(off, 256), 0);
  for (int t = 0; t < T_N; ++t)
    if (src[t].first && src[t].second) std::memcpy(plan->packed.data() + plan->packed_off[t], src[t].first, src[t].second);
}

// Device pointers of a packed image placed at mem.
DevImage image_at(const bfs_plan *plan, void *mem, int dev) {
  DevImage img;
  img.device = dev;
  auto at = [&](int t) { return reinterpret_cast<unsigned char *>(mem) + plan->packed_off[t]; };
  img.code = reinterpret_cast<int32_t *>(at(T_CODE));
  img.code_off = reinterpret_cast<int32_t *>(at(T_COFF));
  img.waits = reinterpret_cast<DevWait *>(at(T_WAIT));
  img.instr_opcode = reinterpret_cast<int32_t *>(at(T_OP));
  img.instr_args = reinterpret_cast<int32_t *>(at(T_ARGS));
  img.instr_waits = reinterpret_cast<int32_t *>(at(T_IW));
  img.waits_by_instr = reinterpret_cast<int32_t *>(at(T_WL));
  img.instr_update = reinterpret_cast<int32_t *>(at(T_UPD));
  img.loop_parent = reinterpret_cast<int32_t *>(at(T_LP));
  img.err = reinterpret_cast<uint32_t *>(mem);
  return img;
}

// ---------------------------------------------------------------------------
// The fixed device array of bfs_run_noalloc.  It holds a plan image (error
// words, then the tables) like the allocation of bfs_run.  Each device keeps
// its own copy at its own address, obtained with hipGetSymbolAddress; host
// code uses that address, never the array's name.  Zero-initialized when the
// code object is loaded; bfs_run_status clears the error words it reports.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = BFS_NOALLOC_MAX_IMAGE_BYTES;

constexpr int kMaxDevices = 64;
struct ScratchDev {
  void *ptr = nullptr;       // device address of this device's copy of scratch
  uint64_t tables_of = 0;    // uid of the plan whose tables it holds (0: none)
};
std::mutex g_scratch_mu;
ScratchDev g_scratch[kMaxDevices];

// Address of the current device's copy (looked up once per device, with the
// device current).  Caller holds g_scratch_mu.
bfs_status scratch_ptr(int dev, void **out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(BFS_E_DEVICE, "device index beyond 64");
  if (!g_scratch[dev].ptr) {
    void *p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(BFS_E_DEVICE, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_scratch[dev].ptr = p;
  }
  *out = g_scratch[dev].ptr;
  return BFS_OK;
}

}  // namespace

bfs_status device_image(const bfs_plan *cplan, DevImage **out) {
  bfs_plan *plan = const_cast<bfs_plan *>(cplan);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("hipGetDevice: ") + hipGetErrorString(e));
  std::lock_guard<std::mutex> lk(plan->dev_mu);
  for (auto &img : plan->images)
    if (img.device == dev) {
      *out = &img;
      return BFS_OK;
    }
  // Every table in one allocation.
  pack_tables(plan);
  void *mem = nullptr;
  e = hipMalloc(&mem, plan->packed.size());
  if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("hipMalloc: ") + hipGetErrorString(e));
  e = hipMemcpy(mem, plan->packed.data(), plan->packed.size(), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(mem);
    return fail(BFS_E_DEVICE, std::string("hipMemcpy: ") + hipGetErrorString(e));
  }
  DevImage img = image_at(plan, mem, dev);
  img.mem = mem;
  plan->images.push_back(img);
  *out = &plan->images.back();
  return BFS_OK;
}

void free_images(bfs_plan *plan) {
  std::lock_guard<std::mutex> lk(plan->dev_mu);
  int cur = 0;
  (void)hipGetDevice(&cur);
  for (auto &img : plan->images) {
    if (!img.mem) continue;
    (void)hipSetDevice(img.device);
    (void)hipFree(img.mem);
    img.mem = nullptr;
  }
  (void)hipSetDevice(cur);
  plan->images.clear();
}

}  // namespace bfs

using namespace bfs;

namespace {

// Argument checks and defaults shared by bfs_run and bfs_run_noalloc.
// Returns BFS_OK with *skip set when there is nothing to launch.
bfs_status run_prologue(const bfs_plan *plan, int32_t n_buffers, const void *const *dev_buffers, int32_t n_wg,
                        uint32_t *dev_debug_log, int64_t debug_capacity, const bfs_run_opts *opts, bfs_run_opts &o,
                        bool *skip) {
  *skip = false;
  if (!plan) return fail(BFS_E_INVALID, "null plan");
  if (n_wg < 0) return fail(BFS_E_INVALID, "negative workgroup count");
  if (n_buffers < 0 || (n_buffers > 0 && !dev_buffers)) return fail(BFS_E_INVALID, "bad buffer list");
  if (dev_debug_log && debug_capacity < 0) return fail(BFS_E_INVALID, "negative debug capacity");
  o = bfs_run_opts{};
  o.watchdog_polls = 1ull << 24;
  o.fault_dep = -1;
  o.fault_delta = 0;
  o.dev_stats = nullptr;
  o.k_unroll = 1;
  o.flags = 0;
  if (opts) {
    if (opts->watchdog_polls) o.watchdog_polls = opts->watchdog_polls;
    o.fault_dep = opts->fault_dep;
    o.fault_delta = opts->fault_delta;
    o.dev_stats = opts->dev_stats;
    if (opts->k_unroll > 1) o.k_unroll = opts->k_unroll;
    if (opts->k_unroll < 0 || (o.k_unroll != 1 && o.k_unroll != 2 && o.k_unroll != 4 && o.k_unroll != 8))
      return fail(BFS_E_INVALID, "k_unroll must be 0, 1, 2, 4 or 8");
    if (opts->flags & ~(BFS_RUN_PER_INSTANCE | BFS_RUN_LOG_BATCHED))
      return fail(BFS_E_INVALID, "unknown bfs_run_opts.flags bits");
    o.flags = opts->flags;
  }
  if (plan->mode == BFS_MODE_BARRIER_FREE && plan->stats.n_fallback > 0 && plan->kernel != BFS_KERNEL_INTERP)
    return fail(BFS_E_UNSUPPORTED, "barrier-fallback dependencies run on the interpreter family only");
  if (plan->mode == BFS_MODE_BARRIER_FREE && plan->alloc == BFS_ALLOC_PER_ENGINE && plan->kernel != BFS_KERNEL_INTERP)
    return fail(BFS_E_UNSUPPORTED, "per-engine allocation runs on the interpreter family only");
  if (n_wg == 0) *skip = true;
  return BFS_OK;
}

bfs_status dispatch(const bfs_plan *plan, DevImage *img, const void *const *dev_buffers, int32_t n_buffers,
                    const int32_t *dev_trips, const int64_t *dev_trip_off, int32_t n_wg, struct ihipStream_t *stream,
                    uint32_t *dev_debug_log, int64_t debug_capacity, const bfs_run_opts &o) {
  switch (plan->kernel) {
    case BFS_KERNEL_INTERP:
      return launch_interp(plan, img, dev_buffers, n_buffers, dev_trips, dev_trip_off, n_wg, stream,
                           dev_debug_log, debug_capacity, o);
    case BFS_KERNEL_STREAM3:
      return launch_stream3(plan, img, dev_buffers, n_buffers, dev_trips, dev_trip_off, n_wg, stream,
                            dev_debug_log, debug_capacity, o);
    case BFS_KERNEL_GEMM:
      return launch_gemm(plan, img, dev_buffers, n_buffers, dev_trips, dev_trip_off, n_wg, stream,
                         dev_debug_log, debug_capacity, o);
    case BFS_KERNEL_ATTN:
      return launch_attn(plan, img, dev_buffers, n_buffers, dev_trips, dev_trip_off, n_wg, stream,
                         dev_debug_log, debug_capacity, o);
    case BFS_KERNEL_ADAMW:
      return launch_adamw(plan, img, dev_buffers, n_buffers, dev_trips, dev_trip_off, n_wg, stream,
                          dev_debug_log, debug_capacity, o);
    case BFS_KERNEL_RMSNORM:
      return launch_rms(plan, img, dev_buffers, n_buffers, dev_trips, dev_trip_off, n_wg, stream,
                        dev_debug_log, debug_capacity, o);
    case BFS_KERNEL_MOE:
      return launch_moe(plan, img, dev_buffers, n_buffers, dev_trips, dev_trip_off, n_wg, stream,
                        dev_debug_log, debug_capacity, o);
    case BFS_KERNEL_CHAIN:
      return launch_chain(plan, img, dev_buffers, n_buffers, dev_trips, dev_trip_off, n_wg, stream,
                          dev_debug_log, debug_capacity, o);
    default:
      return fail(BFS_E_UNSUPPORTED, "kernel family not built");
  }
}

// Reports (and clears) the first error recorded in an image's error words.
bfs_status report_error_words(uint32_t *dev_err) {
  uint32_t w[8] = {0};
  hipError_t e = hipMemcpy(w, dev_err, sizeof w, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("hipMemcpy: ") + hipGetErrorString(e));
  if (w[0] == 0) return BFS_OK;
  uint32_t z[8] = {0};
  (void)hipMemcpy(dev_err, z, sizeof z, hipMemcpyHostToDevice);
  if (w[0] == 2) {
    static const char *what[5] = {"?", "trip count beyond the work item", "trip table disagrees with a static loop",
                                  "load offset beyond 32 bits",
                                  "trip count beyond the ring reuse the program's dependencies order"};
    return fail(BFS_E_INVALID, std::string("run-time input rejected in workgroup ") + std::to_string(w[2]) +
                                   " (wave " + std::to_string(w[6]) + "): " + what[w[1] < 5 ? w[1] : 0] +
                                   " (index " + std::to_string(w[3]) + ", value " + std::to_string(w[4]) +
                                   ", limit " + std::to_string(w[5]) + ")");
  }
  return fail(BFS_E_DEADLOCK, "wait of dependency " + std::to_string(w[1]) + " in workgroup " +
                                  std::to_string(w[2]) + " (wave " + std::to_string(w[6]) + ", instance " +
                                  std::to_string(w[3]) + ") saw " + std::to_string(w[5]) + " < threshold " +
                                  std::to_string(w[4]));
}

}  // namespace

extern "C" {

bfs_status bfs_run(const bfs_plan *plan, const void *const *dev_buffers, int32_t n_buffers,
                   const int32_t *dev_trips, const int64_t *dev_trip_off, int32_t n_wg,
                   struct ihipStream_t *stream, uint32_t *dev_debug_log, int64_t debug_capacity,
                   const bfs_run_opts *opts) {
  bfs_run_opts o;
  bool skip = false;
  bfs_status st = run_prologue(plan, n_buffers, dev_buffers, n_wg, dev_debug_log, debug_capacity, opts, o, &skip);
  if (st != BFS_OK || skip) return st;
  DevImage *img = nullptr;
  st = device_image(plan, &img);
  if (st != BFS_OK) return st;
  return dispatch(plan, img, dev_buffers, n_buffers, dev_trips, dev_trip_off, n_wg, stream, dev_debug_log,
                  debug_capacity, o);
}

bfs_status bfs_run_noalloc(const bfs_plan *cplan, const void *const *dev_buffers, int32_t n_buffers,
                           const int32_t *dev_trips, const int64_t *dev_trip_off, int32_t n_wg,
                           struct ihipStream_t *stream, uint32_t *dev_debug_log, int64_t debug_capacity,
                           const bfs_run_opts *opts) {
  bfs_run_opts o;
  bool skip = false;
  bfs_status st = run_prologue(cplan, n_buffers, dev_buffers, n_wg, dev_debug_log, debug_capacity, opts, o, &skip);
  if (st != BFS_OK || skip) return st;
  bfs_plan *plan = const_cast<bfs_plan *>(cplan);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("hipGetDevice: ") + hipGetErrorString(e));
  DevImage img;
  {
    std::lock_guard<std::mutex> lk(plan->dev_mu);
    pack_tables(plan);
    if (plan->packed.size() > kScratchBytes)
      return fail(BFS_E_RESOURCE, "plan image of " + std::to_string(plan->packed.size()) +
                                      " bytes exceeds the no-allocation limit of " + std::to_string(kScratchBytes));
    std::lock_guard<std::mutex> gk(g_scratch_mu);
    void *mem = nullptr;
    st = scratch_ptr(dev, &mem);
    if (st != BFS_OK) return st;
    // Only the interpreter reads the tables; the other families read the
    // error words alone.  The error words are never overwritten here, so an
    // error stays until bfs_run_status reports it.
    if (plan->kernel == BFS_KERNEL_INTERP && g_scratch[dev].tables_of != plan->uid) {
      e = hipMemcpyAsync(reinterpret_cast<unsigned char *>(mem) + kErrBytes, plan->packed.data() + kErrBytes,
                         plan->packed.size() - kErrBytes, hipMemcpyHostToDevice, (hipStream_t)stream);
      if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("hipMemcpyAsync: ") + hipGetErrorString(e));
      g_scratch[dev].tables_of = plan->uid;
    }
    plan->noalloc_devices |= 1ull << dev;
    img = image_at(plan, mem, dev);
  }
  return dispatch(plan, &img, dev_buffers, n_buffers, dev_trips, dev_trip_off, n_wg, stream, dev_debug_log,
                  debug_capacity, o);
}

bfs_status bfs_run_status(const bfs_plan *cplan, struct ihipStream_t *stream) {
  if (!cplan) return fail(BFS_E_INVALID, "null plan");
  hipError_t e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("hipStreamSynchronize: ") + hipGetErrorString(e));
  if (cplan->mode == BFS_MODE_BARRIER_FREE && cplan->stats.n_fallback > 0 && cplan->kernel != BFS_KERNEL_INTERP)
    return fail(BFS_E_UNSUPPORTED, "barrier-fallback dependencies run on the interpreter family only");
  bfs_plan *plan = const_cast<bfs_plan *>(cplan);
  int dev = 0;
  e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("hipGetDevice: ") + hipGetErrorString(e));
  uint32_t *own = nullptr, *fixed = nullptr;
  {
    std::lock_guard<std::mutex> lk(plan->dev_mu);
    for (auto &img : plan->images)
      if (img.device == dev) own = img.err;
    if (dev >= 0 && dev < kMaxDevices && (plan->noalloc_devices >> dev) & 1ull) {
      std::lock_guard<std::mutex> gk(g_scratch_mu);
      fixed = static_cast<uint32_t *>(g_scratch[dev].ptr);
    }
  }
  if (own) {
    bfs_status st = report_error_words(own);
    if (st != BFS_OK) return st;
  }
  if (fixed) return report_error_words(fixed);
  return BFS_OK;
}

}  // extern "C"
