// Launch-side runtime: per-device plan images, family dispatch and the
// watchdog status word.
#include <hip/hip_runtime.h>

#include <cstring>
#include <string>
#include <vector>

#include "bfs_internal.h"

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
    }
    w[d] = x;
  }
  return w;
}

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
  // Pack every table into one allocation.
  const std::vector<DevWait> waits = device_waits(plan);
  struct Part { const void *src; size_t bytes; size_t off; };
  std::vector<Part> parts;
  size_t off = 0;
  auto add = [&](const void *src, size_t bytes) {
    off = align_up(off, 256);
    parts.push_back(Part{src, bytes, off});
    off += bytes > 0 ? bytes : 4;
    return parts.size() - 1;
  };
  size_t i_code = add(plan->code.data(), plan->code.size() * 4);
  size_t i_coff = add(plan->code_off.data(), plan->code_off.size() * 4);
  size_t i_wait = add(waits.data(), waits.size() * sizeof(DevWait));
  size_t i_op = add(plan->instr_opcode.data(), plan->instr_opcode.size() * 4);
  size_t i_args = add(plan->instr_args.data(), plan->instr_args.size() * 4);
  size_t i_iw = add(plan->instr_wait_off.data(), plan->instr_wait_off.size() * 4);
  size_t i_wl = add(plan->instr_wait_list.data(), plan->instr_wait_list.size() * 4);
  size_t i_upd = add(plan->instr_update.data(), plan->instr_update.size() * 4);
  size_t i_lp = add(plan->loop_parent.data(), plan->loop_parent.size() * 4);
  size_t i_err = add(nullptr, 64);
  const size_t total = align_up(off, 256);
  void *mem = nullptr;
  e = hipMalloc(&mem, total);
  if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("hipMalloc: ") + hipGetErrorString(e));
  std::vector<unsigned char> host(total, 0);
  for (auto &pt : parts)
    if (pt.src && pt.bytes) std::memcpy(host.data() + pt.off, pt.src, pt.bytes);
  e = hipMemcpy(mem, host.data(), total, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(mem);
    return fail(BFS_E_DEVICE, std::string("hipMemcpy: ") + hipGetErrorString(e));
  }
  DevImage img;
  img.device = dev;
  img.mem = mem;
  auto at = [&](size_t i) { return reinterpret_cast<unsigned char *>(mem) + parts[i].off; };
  img.code = reinterpret_cast<int32_t *>(at(i_code));
  img.code_off = reinterpret_cast<int32_t *>(at(i_coff));
  img.waits = reinterpret_cast<DevWait *>(at(i_wait));
  img.instr_opcode = reinterpret_cast<int32_t *>(at(i_op));
  img.instr_args = reinterpret_cast<int32_t *>(at(i_args));
  img.instr_waits = reinterpret_cast<int32_t *>(at(i_iw));
  img.waits_by_instr = reinterpret_cast<int32_t *>(at(i_wl));
  img.instr_update = reinterpret_cast<int32_t *>(at(i_upd));
  img.loop_parent = reinterpret_cast<int32_t *>(at(i_lp));
  img.err = reinterpret_cast<uint32_t *>(at(i_err));
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

extern "C" {

bfs_status bfs_run(const bfs_plan *plan, const void *const *dev_buffers, int32_t n_buffers,
                   const int32_t *dev_trips, const int64_t *dev_trip_off, int32_t n_wg,
                   struct ihipStream_t *stream, uint32_t *dev_debug_log, int64_t debug_capacity,
                   const bfs_run_opts *opts) {
  if (!plan) return fail(BFS_E_INVALID, "null plan");
  if (n_wg < 0) return fail(BFS_E_INVALID, "negative workgroup count");
  if (n_buffers < 0 || (n_buffers > 0 && !dev_buffers)) return fail(BFS_E_INVALID, "bad buffer list");
  if (dev_debug_log && debug_capacity < 0) return fail(BFS_E_INVALID, "negative debug capacity");
  if (n_wg == 0) return BFS_OK;
  bfs_run_opts o{};
  o.watchdog_polls = 1ull << 24;
  o.fault_dep = -1;
  o.fault_delta = 0;
  o.dev_stats = nullptr;
  o.k_unroll = 1;
  if (opts) {
    if (opts->watchdog_polls) o.watchdog_polls = opts->watchdog_polls;
    o.fault_dep = opts->fault_dep;
    o.fault_delta = opts->fault_delta;
    o.dev_stats = opts->dev_stats;
    if (opts->k_unroll > 1) o.k_unroll = opts->k_unroll;
    if (opts->k_unroll < 0 || (o.k_unroll != 1 && o.k_unroll != 2 && o.k_unroll != 4 && o.k_unroll != 8))
      return fail(BFS_E_INVALID, "k_unroll must be 0, 1, 2, 4 or 8");
  }
  if (plan->mode == BFS_MODE_BARRIER_FREE && plan->stats.n_fallback > 0 && plan->kernel != BFS_KERNEL_INTERP)
    return fail(BFS_E_UNSUPPORTED, "barrier-fallback dependencies run on the interpreter family only");
  DevImage *img = nullptr;
  bfs_status st = device_image(plan, &img);
  if (st != BFS_OK) return st;
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
    default:
      return fail(BFS_E_UNSUPPORTED, "kernel family not built");
  }
}

bfs_status bfs_run_status(const bfs_plan *plan, struct ihipStream_t *stream) {
  if (!plan) return fail(BFS_E_INVALID, "null plan");
  hipError_t e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("hipStreamSynchronize: ") + hipGetErrorString(e));
  if (plan->mode == BFS_MODE_BARRIER_FREE && plan->stats.n_fallback > 0 && plan->kernel != BFS_KERNEL_INTERP)
    return fail(BFS_E_UNSUPPORTED, "barrier-fallback dependencies run on the interpreter family only");
  DevImage *img = nullptr;
  bfs_status st = device_image(plan, &img);
  if (st != BFS_OK) return st;
  uint32_t w[8] = {0};
  e = hipMemcpy(w, img->err, sizeof w, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("hipMemcpy: ") + hipGetErrorString(e));
  if (w[0] != 0) {
    uint32_t z[8] = {0};
    (void)hipMemcpy(img->err, z, sizeof z, hipMemcpyHostToDevice);
    if (w[0] == 2) {
      static const char *what[4] = {"?", "trip count beyond the work item", "trip table disagrees with a static loop",
                                    "load offset beyond 32 bits"};
      return fail(BFS_E_INVALID, std::string("run-time input rejected in workgroup ") + std::to_string(w[2]) +
                                     " (wave " + std::to_string(w[6]) + "): " + what[w[1] < 4 ? w[1] : 0] +
                                     " (index " + std::to_string(w[3]) + ", value " + std::to_string(w[4]) +
                                     ", limit " + std::to_string(w[5]) + ")");
    }
    return fail(BFS_E_DEADLOCK, "wait of dependency " + std::to_string(w[1]) + " in workgroup " +
                                    std::to_string(w[2]) + " (wave " + std::to_string(w[6]) + ", instance " +
                                    std::to_string(w[3]) + ") saw " + std::to_string(w[5]) + " < threshold " +
                                    std::to_string(w[4]));
  }
  return BFS_OK;
}

}  // extern "C"
