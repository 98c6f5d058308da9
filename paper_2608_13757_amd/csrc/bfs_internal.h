// Internal definitions shared by the planner and the launch code of libbfs.
#pragma once

#include <cstdint>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/bfs.h"

namespace bfs {

constexpr int kMaxEngines = 8;
constexpr int kMaxLoops = 32;
constexpr int kMaxWavesPerEngine = 8;
constexpr int kMaxWaves = 16;     // waves of one workgroup in the interpreter
constexpr int kMaxSlots = 64;     // counter slots

// Interpreter code words (one engine's projection of the statement tree).
// Per-engine allocation adds TRACK (a0 producer engine, a1 instructions of
// that engine passed in program order) and SNAP (a0 dependency: record the
// producer engine's running count after the producer's position).
enum : int32_t { CODE_LOOP = 1, CODE_END = 2, CODE_INSTR = 3, CODE_HALT = 4, CODE_TRACK = 5, CODE_SNAP = 6 };

// One wait as the device evaluates it.  Barrier-free: Eq. 5 on the consumer
// engine's registers; barrier mode: a static ordinal on the producer engine's
// region counter.
struct DevWait {
  int32_t dep;
  int32_t counter;      // LDS counter slot (barrier mode: producer engine)
  int32_t prd_engine;
  int32_t loop_S;
  int32_t loop_P;
  int32_t k;
  int32_t expr_sub;
  int32_t N;
  int32_t K;
  int32_t needs_mask;
  int32_t ordinal;      // barrier mode
  int32_t active;       // 0: no wait is needed (barrier mode, cross-region)
  int32_t snap_slots;   // per-engine: snapshots kept (0: not per-engine)
  int32_t snap_off;     // per-engine: first snapshot word in the consumer wave's area
  int32_t linear;       // offset read over all trips of S (no mask)
  int32_t pad;
};

// A wait packed into four words for kernels that carry their waits as
// launch arguments:
//   w0 = counter | loop_P << 8 | loop_S << 16 | needs_mask << 24 | active << 25
//   w1 = N | K << 16;  w2 = k | expr_sub << 16;  w3 = dep | ordinal << 16
struct PackedWait {
  uint32_t w0, w1, w2, w3;
};

inline bool pack_wait(const DevWait &d, PackedWait &out) {
  if (d.counter < 0 || d.counter > 255 || d.loop_P > 255 || d.loop_S > 255 || d.N > 65535 || d.K > 65535 ||
      d.k > 65535 || d.expr_sub > 65535 || d.dep > 65535 || d.ordinal > 65535)
    return false;
  out.w0 = (uint32_t)d.counter | (uint32_t)d.loop_P << 8 | (uint32_t)d.loop_S << 16 |
           (uint32_t)(d.needs_mask ? 1 : 0) << 24 | (uint32_t)(d.active ? 1 : 0) << 25;
  out.w1 = (uint32_t)d.N | (uint32_t)d.K << 16;
  out.w2 = (uint32_t)d.k | (uint32_t)d.expr_sub << 16;
  out.w3 = (uint32_t)d.dep | (uint32_t)d.ordinal << 16;
  return true;
}

struct DevImage {
  int device = -1;
  void *mem = nullptr;          // one allocation holding everything below
  int32_t *code = nullptr;      // int32 x4 per word
  int32_t *code_off = nullptr;  // [n_engines + 1] in words
  DevWait *waits = nullptr;
  int32_t *instr_opcode = nullptr;
  int32_t *instr_args = nullptr;
  int32_t *instr_waits = nullptr;  // CSR [n_instrs + 1] into waits_by_instr
  int32_t *waits_by_instr = nullptr;
  int32_t *instr_update = nullptr; // counter slot each instruction increments, -1 none
  int32_t *loop_parent = nullptr;
  uint32_t *err = nullptr;         // watchdog word: [code, dep, wg, instance, thr, observed, wave, pad]
};

bfs_status launch_gemm(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                       const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream,
                       uint32_t *dbg, int64_t dbg_cap, const bfs_run_opts &o);
}  // namespace bfs

struct bfs_plan {
  bfs_mode mode;
  bfs_alloc alloc;
  int32_t kernel;
  int32_t n_engines;
  int32_t waves_per_engine[bfs::kMaxEngines];
  int32_t n_loops;
  std::vector<int32_t> loop_parent, loop_is_cond;
  std::vector<int32_t> body_off, body_kind, body_id;
  std::vector<int32_t> block_off, block_instrs;
  std::vector<int32_t> instr_engine, instr_opcode, instr_args;
  std::vector<int32_t> deps;
  std::vector<int32_t> dep_linear;       // per dependency: 1 = linearized offset (extension)
  int32_t tile_elems;
  int32_t ring_slots[4];
  int32_t n_accs;
  uint32_t flags = 0;                    // bfs_plan_create flags

  // derived structure
  std::vector<int32_t> instr_parent;     // innermost enclosing loop
  std::vector<int32_t> loop_depth;
  // planning results
  std::vector<bfs_formula> formulas;
  std::vector<bfs_static_wait> static_waits;
  std::vector<int32_t> instr_update;     // counter slot incremented at retirement (-1: none)
  int32_t n_counters = 0;
  uint32_t fallback_loops = 0;           // bit l: drain barrier at the end of every iteration of loop l
  bfs_stats stats{};
  // per-instruction wait lists (dependency ids whose consumer is the instruction)
  std::vector<int32_t> instr_wait_off, instr_wait_list;
  // interpreter code (int32 x4 words), per engine
  std::vector<int32_t> code, code_off;
  // per-engine allocation: first snapshot word of each dependency in its
  // consumer engine's area, and the largest area (words)
  std::vector<int32_t> snap_off;
  int32_t snap_words = 0;

  std::mutex dev_mu;
  std::vector<bfs::DevImage> images;     // one per device used
  // bfs_run_noalloc: the packed tables (built once, kept for the
  // asynchronous copies into the static device array), the plan's unique id,
  // and the devices whose static array this plan has written (bit d).
  std::vector<unsigned char> packed;
  std::vector<size_t> packed_off;        // table offsets in `packed`
  uint64_t uid = 0;
  uint64_t noalloc_devices = 0;
};

namespace bfs {
std::vector<DevWait> device_waits(const bfs_plan *p);
void set_error(const std::string &msg);
bfs_status fail(bfs_status s, const std::string &msg);
// Device image of a plan for the current device (uploads on first use).
bfs_status device_image(const bfs_plan *plan, DevImage **out);
void free_images(bfs_plan *plan);
// Family launchers (defined in the .hip files).
bfs_status launch_interp(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                         const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream,
                         uint32_t *dbg, int64_t dbg_cap, const bfs_run_opts &o);
bfs_status launch_stream3(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                          const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream,
                          uint32_t *dbg, int64_t dbg_cap, const bfs_run_opts &o);
bfs_status launch_gemm(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                       const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream,
                       uint32_t *dbg, int64_t dbg_cap, const bfs_run_opts &o);
bfs_status launch_attn(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                       const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream,
                       uint32_t *dbg, int64_t dbg_cap, const bfs_run_opts &o);
bfs_status launch_moe(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                       const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream,
                       uint32_t *dbg, int64_t dbg_cap, const bfs_run_opts &o);
bfs_status launch_rms(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                      const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream,
                      uint32_t *dbg, int64_t dbg_cap, const bfs_run_opts &o);
bfs_status launch_adamw(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                        const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream,
                        uint32_t *dbg, int64_t dbg_cap, const bfs_run_opts &o);
bfs_status launch_chain(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                        const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream,
                        uint32_t *dbg, int64_t dbg_cap, const bfs_run_opts &o);
}  // namespace bfs
