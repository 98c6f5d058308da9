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

#include <initializer_list>
#include <string>
#include <utility>
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

// How a wait's threshold moves while the consumer's innermost loop L runs
// (decided on the host from the loop tree):
//   affine   producer and shared loop are L itself (C1 at L): Eq. 5 is
//            base + N * rhat_L with the mask rhat_L > k, base fixed at L's entry;
//   constant the producer's loop lies outside L's subtree and the shared loop
//            is a proper ancestor of L: Eq. 5 does not change during L's trip
//            (and in barrier mode every threshold is a constant ordinal);
//   dynamic  the producer's loop is nested inside L or the shared loop is L
//            with an outer producer: Eq. 5 is evaluated at every wait.
constexpr int32_t kWaitAffine = 0, kWaitConst = 1, kWaitDynamic = 2;

struct Wait {
  bfs::PackedWait w;
  int32_t n_prd_waves;
  int32_t kind;
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
// Selection by bit masks keeps the registers in scalar registers (a
// conditional chain is turned into a stack lookup table by the compiler).
struct Regs {
  uint32_t r1 = 0, r2 = 0, r3 = 0, h1 = 0, h2 = 0, h3 = 0;
  __device__ __forceinline__ static uint32_t sel(uint32_t l, uint32_t v1, uint32_t v2, uint32_t v3) {
    const uint32_t m0 = 0u - (uint32_t)(l == 0), m1 = 0u - (uint32_t)(l == 1);
    const uint32_t m2 = 0u - (uint32_t)(l == 2), m3 = 0u - (uint32_t)(l == 3);
    return (m0 & 1u) | (m1 & v1) | (m2 & v2) | (m3 & v3);
  }
  __device__ __forceinline__ uint32_t r(uint32_t l) const { return sel(l, r1, r2, r3); }
  __device__ __forceinline__ uint32_t h(uint32_t l) const { return sel(l, h1, h2, h3); }
};

// The loop-invariant part of one instruction's waits, set up at each entry
// to the instruction's innermost loop (Section 6.2: only the iteration-
// dependent term is evaluated per iteration), plus the monotone "seen" cache.
// kN is the most waits the call site takes (launchers check it).  Per wait:
// meta = counter word address (bits 0-15) | producer waves (16-19) | kind
// (20-21); mk = mask offset k (0-15) | N (16-31); base = the affine or
// constant part of Eq. 5.
template <int kN>
struct Site {
  uint32_t n = 0;
  uint32_t meta[kN];
  uint32_t mk[kN];
  int32_t base[kN];
  uint32_t seen[kN];
  __device__ Site() {
#pragma unroll
    for (int j = 0; j < kN; ++j) {
      meta[j] = 0;
      mk[j] = 0;
      base[j] = 0;
      seen[j] = 0;
    }
  }
};

// Minimum of v over lanes 0 .. 15 with DPP moves (no LDS traffic), read from
// lane 0.  The counter polls put producer wave w's word in lane w and repeat
// lane 0's word in every lane at or above the producer count, so this is the
// minimum over the producer waves.
__device__ __forceinline__ uint32_t min16(uint32_t v) {
  v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false));    // quad_perm 1,0,3,2
  v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false));    // quad_perm 2,3,0,1
  v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x124, 0xF, 0xF, false));   // row_ror 4
  v = min(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x128, 0xF, 0xF, false));   // row_ror 8
  return __builtin_amdgcn_readfirstlane(v);
}

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

  // Poll until every producer word reaches thr; returns the minimum
  // observed producer word.  on_block() runs before every repeated poll: a
  // producer that holds unretired work retires its oldest piece there, one
  // at a time, so the consumers it may be waiting for make progress while
  // its younger loads stay in flight.
  template <class OnBlock>
  __device__ __forceinline__ uint32_t poll_geq(uint32_t addr, uint32_t nw, uint32_t thr, uint32_t dep,
                                               uint32_t instance, OnBlock on_block) {
    if (nw == 1) {
      // one producer wave: a scalar compare of its word
      uint32_t v = uniform(lds_poll(addr));
      if (v >= thr) return v;
      on_block();
      const uint64_t t0 = (kInstr && st.on) ? now_ticks() : 0;
      const uint32_t limit = C.watchdog > 0xffffffffull ? 0xffffffffu : (uint32_t)C.watchdog;
      uint32_t polls = 0;
      while (true) {
        v = uniform(lds_poll(addr));
        if (v >= thr) break;
        on_block();
        if (++polls > limit) {
          report_deadlock(C.err, dep, (uint32_t)wg, instance, thr, v, (uint32_t)wave);
          aborted = 1u;
          return v;
        }
        if (polls < 4) __builtin_amdgcn_s_sleep(1);
        else __builtin_amdgcn_s_sleep(2);
      }
      if (kInstr && st.on) {
        st.blocked += now_ticks() - t0;
        st.n_blocked += 1;
      }
      return v;
    }
    const uint32_t lane = lane_id();
    const uint32_t a = addr + 4u * (lane < nw ? lane : 0u);
    const uint64_t want = (1ull << nw) - 1ull;
    uint32_t v = lds_poll(a);
    if ((__ballot(v >= thr) & want) == want) return min16(v);
    on_block();
    const uint64_t t0 = (kInstr && st.on) ? now_ticks() : 0;
    const uint32_t limit = C.watchdog > 0xffffffffull ? 0xffffffffu : (uint32_t)C.watchdog;
    uint32_t polls = 0;
    while (true) {
      v = lds_poll(a);
      if ((__ballot(v >= thr) & want) == want) break;
      on_block();
      if (++polls > limit) {
        const uint32_t m = min16(v);
        report_deadlock(C.err, dep, (uint32_t)wg, instance, thr, m, (uint32_t)wave);
        aborted = 1u;
        return m;
      }
      if (polls < 4) __builtin_amdgcn_s_sleep(1);
      else __builtin_amdgcn_s_sleep(2);
    }
    if (kInstr && st.on) {
      st.blocked += now_ticks() - t0;
      st.n_blocked += 1;
    }
    return min16(v);
  }

  // Set up the waits of an instruction whose innermost loop is L, before
  // the first iteration of a trip of L (g still holds r_L of the previous
  // trips).
  template <int kN>
  __device__ __forceinline__ void enter(Site<kN> &s, const InstrWaits &iw, const Regs &g, uint32_t L) {
    s.n = (uint32_t)iw.n;
    // Every element is assigned unconditionally (selects, no stores under
    // branches): stores of different elements merged across branches would
    // index the arrays dynamically and move them to scratch memory.
#pragma unroll
    for (int j = 0; j < kN; ++j) {
      const bool on = j < iw.n;
      const bfs::PackedWait w = iw.w[j].w;
      uint32_t kind = (uint32_t)iw.w[j].kind;
      int32_t base = s.base[j];
      uint32_t mk = s.mk[j];
      if (kMode == BFS_MODE_BARRIER) {
        kind = (uint32_t)kWaitConst;
        base = ((w.w0 >> 25) & 1u) ? (int32_t)(w.w3 >> 16) : 0;
      } else {
        const int32_t N = (int32_t)(w.w1 & 0xffffu), K = (int32_t)(w.w1 >> 16);
        const int32_t sub = (int32_t)(w.w2 >> 16);
        const int32_t b_aff = N * ((int32_t)g.r(L) - sub) - (N - K);
        const uint32_t mk_aff = (((w.w0 >> 24) & 1u) ? (w.w2 & 0xffffu) : 0u) | ((uint32_t)N << 16);
        const bool aff = kind == (uint32_t)kWaitAffine, cst = kind == (uint32_t)kWaitConst;
        const int32_t b_cst = cst ? (int32_t)threshold_plain(w, g) : 0;
        base = aff ? b_aff : (cst ? b_cst : base);
        mk = aff ? mk_aff : (cst ? 0u : mk);        // a constant: slope 0, no mask
      }
      const uint32_t meta = word(w.w0 & 0xffu, 0) | ((uint32_t)iw.w[j].n_prd_waves << 16) | (kind << 20);
      s.base[j] = on ? base : s.base[j];
      s.mk[j] = on ? mk : s.mk[j];
      s.meta[j] = on ? meta : s.meta[j];
    }
  }

  // Eq. 5 (no fault injection).
  __device__ __forceinline__ uint32_t threshold_plain(const bfs::PackedWait &w, const Regs &g) const {
    return eq5(g.r((w.w0 >> 8) & 0xffu), g.h((w.w0 >> 16) & 0xffu), (int)(w.w2 & 0xffffu), (int)(w.w2 >> 16),
               (int)(w.w1 & 0xffffu), (int)(w.w1 >> 16), (int)((w.w0 >> 24) & 1u));
  }

  // All waits of the instruction at iteration t (rhat of its loop, from 1).
  template <int kN, class OnBlock>
  __device__ __forceinline__ void wait(Site<kN> &s, const InstrWaits &iw, const Regs &g, uint32_t t,
                                       uint32_t instance, OnBlock on_block) {
#pragma unroll
    for (int j = 0; j < kN; ++j) {
      if ((uint32_t)j < s.n) {
        const uint32_t kind = (s.meta[j] >> 20) & 3u;
        uint32_t thr;
        if (kind == (uint32_t)kWaitAffine) {
          const int32_t v = s.base[j] + (int32_t)((s.mk[j] >> 16) * t);
          thr = (t > (s.mk[j] & 0xffffu) && v > 0) ? (uint32_t)v : 0u;
        } else if (kind == (uint32_t)kWaitConst) {
          thr = (uint32_t)s.base[j];
        } else {
          thr = threshold_plain(iw.w[j].w, g);
        }
        uint32_t dep = 0;
        if (kInstr) {
          dep = iw.w[j].w.w3 & 0xffffu;
          if ((int)dep == C.fault_dep) thr += (uint32_t)C.fault_delta;
        }
        uint32_t obs = kMode == BFS_MODE_BARRIER ? 0u : s.seen[j];
        if (!aborted && thr > 0 && (obs < thr || (kInstr && log))) {
          obs = poll_geq(s.meta[j] & 0xffffu, (s.meta[j] >> 16) & 0xfu, thr,
                         kInstr ? dep : (iw.w[j].w.w3 & 0xffffu), instance, on_block);
          s.seen[j] = obs;
        }
        if (kInstr && log) {
          on_block();
          log_wait(log, C.dbg_cap, nlog, dep, instance, thr, thr > 0 ? obs : 0u);
        }
      }
    }
  }

  // The waits of a site none of whose waits is dynamic (checked on the
  // host): an affine threshold is base + N * t under the mask t > k, a
  // constant one the same with slope 0 and no mask (as enter() stores it),
  // so every wait is evaluated without the per-kind dispatch of wait().
  // Barrier mode and instrumented builds take wait().
  template <int kN, class OnBlock>
  __device__ __forceinline__ void wait_affine(Site<kN> &s, const InstrWaits &iw, const Regs &g, uint32_t t,
                                              uint32_t instance, OnBlock on_block) {
    if constexpr (kMode == BFS_MODE_BARRIER || kInstr) {
      wait(s, iw, g, t, instance, on_block);
    } else {
#pragma unroll
      for (int j = 0; j < kN; ++j) {
        if ((uint32_t)j < s.n) {
          const int32_t v = s.base[j] + (int32_t)((s.mk[j] >> 16) * t);
          const uint32_t thr = (t > (s.mk[j] & 0xffffu) && v > 0) ? (uint32_t)v : 0u;
          if (!aborted && thr > s.seen[j])
            s.seen[j] = poll_geq(s.meta[j] & 0xffffu, (s.meta[j] >> 16) & 0xfu, thr, iw.w[j].w.w3 & 0xffffu,
                                 instance, on_block);
        }
      }
    }
  }

  // One wait whose threshold is a static immediate (straight-line code with
  // no loop register, e.g. an unrolled loop): counter slot `slot` of a
  // producer engine of `nw` waves; `seen` is the caller's monotone cache.
  template <class OnBlock>
  __device__ __forceinline__ void wait_fixed(uint32_t slot, uint32_t nw, uint32_t thr, uint32_t dep, uint32_t instance,
                                             uint32_t &seen, OnBlock on_block) {
    if (kInstr && (int)dep == C.fault_dep) thr += (uint32_t)C.fault_delta;
    uint32_t obs = kMode == BFS_MODE_BARRIER ? 0u : seen;
    if (!aborted && thr > 0 && (obs < thr || (kInstr && log))) {
      obs = poll_geq(word(slot, 0), nw, thr, dep, instance, on_block);
      seen = obs;
    }
    if (kInstr && log) {
      on_block();
      log_wait(log, C.dbg_cap, nlog, dep, instance, thr, thr > 0 ? obs : 0u);
    }
  }

  // Retirement: add 1 to this wave's word of the instruction's counter.
  // LDS executes one wave's DS instructions in issue order, so an add issued
  // after the instruction's LDS writes (its results) and LDS reads (its last
  // use of a slot) takes effect after them: engines whose effects are LDS
  // accesses signal without waiting.  Direct-to-LDS loads are retired by
  // their issuer after a counted vmcnt wait instead.
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
// Host: true when loop x lies in the subtree of loop l (x == l included).
inline bool in_subtree(const bfs_plan *p, int x, int l) {
  for (; x >= 0; x = p->loop_parent[x])
    if (x == l) return true;
  return false;
}

// Host: copy one instruction's waits (and its counter slot) into kernel
// arguments, with each wait's kind relative to the instruction's innermost
// loop.  False when the instruction has more waits than fit.
inline bool fill_waits(const bfs_plan *p, const std::vector<DevWait> &dw, int ins, bfsdev::InstrWaits &out) {
  out.n = 0;
  out.update = p->instr_update[ins];
  const int L = p->instr_parent[ins];
  for (int wi = p->instr_wait_off[ins]; wi < p->instr_wait_off[ins + 1]; ++wi) {
    if (out.n == bfsdev::kMaxWaits) return false;
    const DevWait &d = dw[p->instr_wait_list[wi]];
    if (!pack_wait(d, out.w[out.n].w)) return false;
    out.w[out.n].n_prd_waves = p->waves_per_engine[d.prd_engine];
    int kind = bfsdev::kWaitDynamic;
    if (d.loop_P == L && d.loop_S == L) kind = bfsdev::kWaitAffine;
    else if (!in_subtree(p, d.loop_P, L) && d.loop_S != L) kind = bfsdev::kWaitConst;
    out.w[out.n].kind = kind;
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

// Host: no wait of the instruction is dynamic (each is affine in its
// innermost loop's iteration or constant during its trip), so
// Sync::wait_affine may serve it.
inline bool no_dynamic(const bfsdev::InstrWaits &iw) {
  for (int j = 0; j < iw.n; ++j)
    if (iw.w[j].kind == bfsdev::kWaitDynamic) return false;
  return true;
}

// Host: every instruction's wait count fits its kernel call site.
inline bool waits_fit(std::initializer_list<std::pair<const bfsdev::InstrWaits *, int>> sites) {
  for (auto &x : sites)
    if (x.first->n > x.second) return false;
  return true;
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
