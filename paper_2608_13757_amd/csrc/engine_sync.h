// Engine-side synchronization shared by the fused MFMA kernel families
// (GEMM, attention, MoE): per-instruction wait lists in kernel arguments,
// Eq. 5 thresholds from the engine's loop registers, counter polls with a
// monotone "seen" cache, retirement signals, barrier-mode sync points, the
// debug log and per-wave statistics.
//
// Counter words: slot s, producer wave w at LDS word s * kMaxWavesPerEngine
// + w.  A wait requires every wave of the producer engine to reach the
// threshold.
#pragma once

#include <string>
#include <vector>

#include "bfs_internal.h"
#include "device_sync.h"

namespace bfsdev {

constexpr int kMaxWaits = 4;
constexpr uint32_t kCntBytes = bfs::kMaxSlots * bfs::kMaxWavesPerEngine * 4;

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

struct Wait {
  bfs::PackedWait w;
  int32_t n_prd_waves;
  int32_t pad;
};

// The waits of one instruction and the counter slot it increments.
struct InstrWaits {
  int32_t n;
  int32_t update;          // counter slot, -1 none
  Wait w[kMaxWaits];
};

// Launch-wide instrumentation and error reporting.
struct SyncCommon {
  uint32_t *dbg;           // debug log (null: off)
  int64_t dbg_cap;
  uint32_t *err;           // error word block of the plan image
  uint64_t *stats;         // per-wave statistics (null: off)
  uint64_t watchdog;       // polls before a wait is declared deadlocked
  int32_t fault_dep, fault_delta;
  int32_t n_waves;         // waves per workgroup
  int32_t pad;
};

// Loop registers of a nest with at most three loops below the top level:
// r counts iterations since the start of the workgroup, h (rhat) within the
// current trip (Section 5.1).  The top-level loop runs once.
struct Regs {
  uint32_t r1 = 0, r2 = 0, r3 = 0, h1 = 0, h2 = 0, h3 = 0;
  __device__ __forceinline__ uint32_t r(uint32_t l) const { return l == 0 ? 1u : l == 1 ? r1 : l == 2 ? r2 : r3; }
  __device__ __forceinline__ uint32_t h(uint32_t l) const { return l == 0 ? 1u : l == 1 ? h1 : l == 2 ? h2 : h3; }
};

template <int kMode, bool kInstr>
struct Sync {
  const SyncCommon &C;
  uint32_t cnt_base;
  int wave, wg;            // wave: engine-ordered index (debug log, stats)
  uint32_t aborted = 0;
  uint32_t *log = nullptr;
  uint32_t nlog = 0;
  WaveStats st;

  __device__ Sync(const SyncCommon &c, uint32_t cb, int w, int g) : C(c), cnt_base(cb), wave(w), wg(g) {
    if (kInstr) {
      if (C.dbg) log = C.dbg + (int64_t)gridDim.x * C.n_waves + ((int64_t)wg * C.n_waves + wave) * 4 * C.dbg_cap;
      if (C.stats) {
        st.on = true;
        st.t_start = now_ticks();
      }
    }
  }

  __device__ __forceinline__ uint32_t word(uint32_t slot, uint32_t w) const {
    return cnt_base + 4u * (slot * (uint32_t)bfs::kMaxWavesPerEngine + w);
  }

  __device__ __forceinline__ uint32_t threshold(const bfs::PackedWait &w, const Regs &g) const {
    uint32_t thr;
    if (kMode == BFS_MODE_BARRIER) {
      thr = ((w.w0 >> 25) & 1u) ? (w.w3 >> 16) : 0u;
    } else {
      thr = eq5(g.r((w.w0 >> 8) & 0xffu), g.h((w.w0 >> 16) & 0xffu), (int)(w.w2 & 0xffffu), (int)(w.w2 >> 16),
                (int)(w.w1 & 0xffffu), (int)(w.w1 >> 16), (int)((w.w0 >> 24) & 1u));
    }
    if (kInstr && (int)(w.w3 & 0xffffu) == C.fault_dep) thr += (uint32_t)C.fault_delta;
    return thr;
  }

  // All waits of one instruction.  on_block() retires what this wave holds
  // before it would block.  seen[] keeps, per wait of this instruction, the
  // last counter value observed: counters only grow, so it stays a valid lower
  // bound (barrier mode resets counters, so there every wait polls).
  template <class OnBlock>
  __device__ __forceinline__ void waits(const InstrWaits &iw, const Regs &g, uint32_t instance,
                                        uint32_t (&seen)[kMaxWaits], OnBlock on_block) {
    for (int j = 0; j < iw.n; ++j) {
      const bfs::PackedWait w = iw.w[j].w;
      const int nw = iw.w[j].n_prd_waves;
      const uint32_t thr = threshold(w, g);
      uint32_t obs = kMode == BFS_MODE_BARRIER ? 0u : seen[j];
      if (!aborted && thr > 0 && (obs < thr || (kInstr && log))) {
        const uint32_t a = word(w.w0 & 0xffu, 0);
        WaitResult res = wait_geq(a, nw, thr, 0);   // one poll
        if (!res.ok) {
          on_block();
          const uint64_t t0 = (kInstr && st.on) ? now_ticks() : 0;
          res = wait_geq(a, nw, thr, C.watchdog);
          if (kInstr && st.on) {
            st.blocked += now_ticks() - t0;
            st.n_blocked += 1;
          }
          if (!res.ok) {
            report_deadlock(C.err, w.w3 & 0xffffu, (uint32_t)wg, instance, thr, res.observed, (uint32_t)wave);
            aborted = 1u;
          }
        }
        obs = res.observed;
        seen[j] = obs;
      }
      if (kInstr && log) {
        on_block();
        log_wait(log, C.dbg_cap, nlog, w.w3 & 0xffffu, instance, thr, thr > 0 ? obs : 0u);
      }
    }
  }

  __device__ __forceinline__ void signal(int update, uint32_t ew) {
    if (update >= 0) lds_add(word((uint32_t)update, ew), 1u);
  }

  __device__ __forceinline__ void sync_point(uint32_t own_word) {
    if (kMode == BFS_MODE_BARRIER) {
      const uint64_t t0 = (kInstr && st.on) ? now_ticks() : 0;
      region_sync(own_word, 1);
      if (kInstr && st.on) st.barrier += now_ticks() - t0;
    }
  }

  // o[6] is a free timestamp slot (kernel-defined, e.g. the end of a loop).
  __device__ void finish(uint32_t lane, uint64_t mark = 0) {
    if (!kInstr) return;
    if (C.dbg && lane == 0) C.dbg[(int64_t)wg * C.n_waves + wave] = nlog;
    if (st.on && lane == 0) {
      uint64_t *o = C.stats + ((int64_t)wg * C.n_waves + wave) * 8;
      o[0] = now_ticks() - st.t_start;
      o[1] = st.blocked;
      o[2] = st.n_blocked;
      o[3] = st.barrier;
      o[4] = st.own_loads;
      o[5] = 0;
      o[6] = mark;
      o[7] = 0;
    }
  }

  __device__ __forceinline__ uint64_t elapsed() const { return (kInstr && st.on) ? now_ticks() - st.t_start : 0; }
};

}  // namespace bfsdev

namespace bfs {

// Host: copy one instruction's waits (and its counter slot) into kernel
// arguments.  False when the instruction has more waits than fit.
inline bool fill_waits(const bfs_plan *p, const std::vector<DevWait> &dw, int ins, bfsdev::InstrWaits &out) {
  out.n = 0;
  out.update = p->instr_update[ins];
  for (int wi = p->instr_wait_off[ins]; wi < p->instr_wait_off[ins + 1]; ++wi) {
    if (out.n == bfsdev::kMaxWaits) return false;
    const DevWait &d = dw[p->instr_wait_list[wi]];
    if (!pack_wait(d, out.w[out.n].w)) return false;
    out.w[out.n].n_prd_waves = p->waves_per_engine[d.prd_engine];
    out.n += 1;
  }
  return true;
}

// Host: true when the program lists dependency (prd, cns, k).
inline bool has_dep(const bfs_plan *p, int prd, int cns, int k) {
  for (size_t d = 0; d < p->deps.size() / 3; ++d)
    if (p->deps[3 * d] == prd && p->deps[3 * d + 1] == cns && p->deps[3 * d + 2] == k) return true;
  return false;
}

// Host: launch-wide instrumentation block from the run options.
inline bfsdev::SyncCommon sync_common(const DevImage *img, uint32_t *dbg, int64_t dbg_cap, const bfs_run_opts &o,
                                      int n_waves) {
  bfsdev::SyncCommon c{};
  c.dbg = dbg;
  c.dbg_cap = dbg_cap;
  c.err = img->err;
  c.stats = o.dev_stats;
  c.watchdog = o.watchdog_polls;
  c.fault_dep = o.fault_dep;
  c.fault_delta = o.fault_delta;
  c.n_waves = n_waves;
  return c;
}

}  // namespace bfs
