// Sync-bound stream over a dynamically bounded 3-level nest O{ M{ I{ ... } } }
// with three single-wave engines: E0 loads a 64-element fp32 tile from HBM
// into an LDS ring slot, E1 adds a constant into a second ring, E2 stores the
// result to HBM.  Acquire / marker instructions (no datapath) may sit in the
// bodies of O and M before or after the nested loop.
//
// Waits come from the plan: every instruction evaluates the waits whose
// consumer it is, with Eq. 5 on the engine's loop registers (barrier-free),
// or the static ordinal (barrier mode, which also synchronizes before every
// loop statement and at every iteration end).  The waits of each engine's
// instructions travel in the launch arguments, so the loop body reads no
// descriptor tables.  Each engine runs its own copy of the loop nest, and the
// synchronization mode and the instrumentation are compile-time choices, so
// the innermost loop holds only that engine's work.
//
// Retirement is in issue order:
//   * the load engine keeps up to kInflight direct-to-LDS loads outstanding
//     and retires the oldest with a counted vmcnt wait;
//   * the add engine signals right after its ring write and the store
//     engine right after its ring read returned: LDS executes the operations
//     of one wave in issue order, so the counter add lands after the write;
//   * markers retire at once, after everything before them.
// Before blocking on a wait that is not met, an engine retires what it holds
// (the load engine one load at a time), so a consumer never waits on a
// retirement that the blocked producer is holding back.
//
// Counters only grow, so a counter value an engine has already observed stays
// a valid lower bound: the waits of the innermost instruction remember their
// last observation and poll LDS only when the new threshold exceeds it.
//
// Family contract (BFS_KERNEL_STREAM3): loops top -> O -> M -> I, three
// engines of one wave, tile_elems 64; the I body holds exactly one load
// (engine 0), one add-constant (engine 1) and one store-slot (engine 2), all
// addressed with slot = ((r_M - 1) % n_gen) * per_gen + (rhat_I - 1) % per_gen
// (at most 128 slots per ring, rings 0 and 1; the add may write the ring it
// reads) and tile index base[wg] + r_I - 1.  Buffers: [0] int64 tile base per
// workgroup, [1] fp32 input tiles, [2] fp32 output tiles.
#include <algorithm>
#include <string>

#include "bfs_internal.h"
#include "device_sync.h"

using namespace bfsdev;

namespace {

constexpr int kMaxNops = 4;
constexpr int kMaxWaitsPerEngine = 16;
constexpr int kMaxInnerWaits = 2;
// Batch loads the load engine keeps in flight beyond the one just issued:
// more hides more HBM latency but delays every completion signal by as many
// batches (measured best at 4; 2, 3, 5 and 6 slower).
constexpr uint32_t kBatchQ = 4;

struct InstrSync {
  int16_t first;     // index of its first wait in the engine's wait list
  int16_t n;         // number of waits
  int16_t update;    // counter slot incremented at retirement (-1: none)
  int16_t pad;
};

struct EngineCode {
  InstrSync o_pre[kMaxNops], m_pre[kMaxNops], m_post[kMaxNops], o_post[kMaxNops];
  int32_t n_o_pre, n_m_pre, n_m_post, n_o_post;
  InstrSync inner;
  bfs::PackedWait waits[kMaxWaitsPerEngine];
};

struct Stream3Params {
  EngineCode eng[3];
  const int32_t *trips;
  const int64_t *trip_off;
  const int64_t *base;
  const float *x;
  float *y;
  uint32_t *dbg;
  int64_t dbg_cap;
  uint32_t *err;
  uint64_t *stats;
  uint64_t watchdog;
  int32_t fault_dep, fault_delta;
  int32_t n_gen, per_gen, n_slots;
  int32_t ring_ld, ring_add_src, ring_add_dst, ring_st;   // ring id of each access
  float addc;
  // Largest trips of M and I whose ring-slot reuse the program's
  // dependencies order (derived on the host); longer trips are reported as
  // invalid input and clamped, identically by every engine.
  uint32_t max_trip_m, max_trip_i;
  int32_t per_instance;    // uninstrumented barrier-free: every trip of I on the per-instance loop
  int32_t log_batched;     // instrumented barrier-free: log from the batched loop
};

// The launch arguments are read in place from the kernel-argument segment
// (scalar loads, also at run-time indices) through references of this type.
// (The host pass of the compiler, which only parses device code, sees plain
// const references.)
#if defined(__HIP_DEVICE_COMPILE__)
template <typename T>
using kconst = const __attribute__((address_space(4))) T;
#else
template <typename T>
using kconst = const T;
#endif

__device__ __forceinline__ uint32_t sel4(uint32_t a, uint32_t b, uint32_t c, uint32_t d, uint32_t i) {
  return i == 0 ? a : i == 1 ? b : i == 2 ? c : d;
}

enum { ROLE_LOAD = 0, ROLE_ADD = 1, ROLE_STORE = 2 };

typedef float f32x4 __attribute__((ext_vector_type(4)));

// One engine wave: loop registers, counters, waits and retirement.
template <int kRole, int kMode, bool kInstr, int kInflight>
struct Engine {
  kconst<Stream3Params> &P;
  kconst<EngineCode> &C;
  uint32_t r1 = 0, r2 = 0, r3 = 0;        // r of O, M, I (r of the top level is 1)
  uint32_t h1 = 0, h2 = 0, h3 = 0;        // rhat of O, M, I
  uint32_t cnt_base;
  int wave, wg;
  uint32_t aborted = 0;                   // a wait gave up: finish without waiting
  uint32_t *log = nullptr;
  uint32_t nlog = 0;
  int pending = 0;                        // load engine: loads issued, not yet retired
  // Load engine batches: the tile counts of the last kBatchQ batches issued,
  // oldest first, in scalar registers (0 once retired).
  uint32_t q[kBatchQ] = {};
  // Retirement add with every lane active: lane 0 adds to the inner
  // instruction's counter (or to its own scratch word when the instruction
  // has no consumer), the other lanes add 0 to this wave's private scratch
  // words, so no exec-mask save / restore or branch is needed around the add.
  uint32_t own_vaddr = 0, one_v = 0, scratch_v = 0;
  WaveStats st;

  __device__ Engine(kconst<Stream3Params> &p, kconst<EngineCode> &c, uint32_t cb, int w, int g)
      : P(p), C(c), cnt_base(cb), wave(w), wg(g) {}

  __device__ __forceinline__ void add_own(uint32_t n) {
    // (a constant 1 uses the value prepared at the start; any other count
    // is selected into lane 0 here)
    const uint32_t v = (__builtin_constant_p(n) && n == 1u) ? one_v : (lane_id() == 0 ? n : 0u);
    asm volatile("ds_add_u32 %0, %1" ::"v"(own_vaddr), "v"(v) : "memory");
  }
  __device__ __forceinline__ void add_one(uint32_t addr) {
    const uint32_t a = lane_id() == 0 ? addr : scratch_v;
    asm volatile("ds_add_u32 %0, %1" ::"v"(a), "v"(one_v) : "memory");
  }

  __device__ __forceinline__ uint32_t counter_addr(uint32_t slot) const {
    return cnt_base + 4u * slot * (uint32_t)bfs::kMaxWavesPerEngine;
  }

  __device__ __forceinline__ uint32_t threshold(const bfs::PackedWait &w) const {
    uint32_t thr;
    if (kMode == BFS_MODE_BARRIER) {
      thr = ((w.w0 >> 25) & 1u) ? (w.w3 >> 16) : 0u;
    } else {
      const uint32_t lp = (w.w0 >> 8) & 0xffu, ls = (w.w0 >> 16) & 0xffu;
      const uint32_t rP = sel4(1u, r1, r2, r3, lp), hS = sel4(1u, h1, h2, h3, ls);
      thr = eq5(rP, hS, (int)(w.w2 & 0xffffu), (int)(w.w2 >> 16), (int)(w.w1 & 0xffffu), (int)(w.w1 >> 16),
                (int)((w.w0 >> 24) & 1u));
    }
    if (kInstr && (int)(w.w3 & 0xffffu) == P.fault_dep) thr += (uint32_t)P.fault_delta;
    return thr;
  }

  // --- retirement of the inner instruction --------------------------------
  // Load engine: the oldest of kInflight outstanding loads.
  __device__ __forceinline__ void retire_oldest_of_full() {
    const uint64_t t0 = (kInstr && st.on) ? now_ticks() : 0;
    wait_vm<kInflight - 1>();
    if (kInstr && st.on) st.own_loads += now_ticks() - t0;
    add_own(1u);
    pending = (int)uniform((uint32_t)pending - 1u);
  }
  // Load engine: retire every outstanding batch load.
  __device__ __forceinline__ void flush_batches() {
    if (kRole == ROLE_LOAD) {
      uint32_t held = 0;
#pragma unroll
      for (int i = 0; i < (int)kBatchQ; ++i) held += q[i];
      if (held != 0u) {
        wait_vm<0>();
        add_own(held);
#pragma unroll
        for (int i = 0; i < (int)kBatchQ; ++i) q[i] = 0;
      }
    }
  }
  // Load engine: batch b of k tiles was issued; the batch issued kBatchQ
  // batches earlier retires (entries of batches already flushed are 0).
  __device__ __forceinline__ void issued_batch(uint32_t k) {
    const uint32_t t = q[0];
#pragma unroll
    for (int i = 0; i + 1 < (int)kBatchQ; ++i) q[i] = q[i + 1];
    q[kBatchQ - 1] = k;
    wait_vm<kBatchQ>();
    add_own(t);
  }
  // Retire everything held.
  __device__ __forceinline__ void retire_all() {
    flush_batches();
    if (pending > 0) {
      if (kRole == ROLE_LOAD) {
        const uint64_t t0 = (kInstr && st.on) ? now_ticks() : 0;
        wait_vm<0>();
        if (kInstr && st.on) st.own_loads += now_ticks() - t0;
      } else {
        drain_lds();
      }
      add_own((uint32_t)pending);
      pending = 0;
    }
  }
  // While blocked: the load engine retires one load at a time, the others
  // everything at once.
  __device__ __forceinline__ void retire_some() {
    if (kRole == ROLE_LOAD) {
      wait_vm_dyn(pending - 1);
      add_own(1u);
      pending -= 1;
    } else {
      retire_all();
    }
  }

  __device__ __forceinline__ WaitResult block(uint32_t addr, uint32_t thr, uint32_t dep, uint32_t instance) {
    const uint64_t t0 = (kInstr && st.on) ? now_ticks() : 0;
    if (kInstr && st.on) st.n_blocked += 1;
    flush_batches();
    while (pending > 0) {
      const uint32_t v = uniform(lds_poll(addr));
      if (v >= thr) {
        if (kInstr && st.on) st.blocked += now_ticks() - t0;
        return WaitResult{v, true};
      }
      retire_some();
    }
    WaitResult res = spin_geq(addr, thr, P.watchdog);
    if (kInstr && st.on) st.blocked += now_ticks() - t0;
    if (!res.ok) {
      report_deadlock(P.err, dep, (uint32_t)wg, instance, thr, res.observed, (uint32_t)wave);
      aborted = 1u;
    }
    return res;
  }

  __device__ __forceinline__ void logit(uint32_t dep, uint32_t instance, uint32_t thr, uint32_t obs) {
    if (kInstr && log) {
      retire_all();   // log stores share vmcnt with the loads
      log_wait(log, P.dbg_cap, nlog, dep, instance, thr, obs);
    }
  }

  // One wait: returns the observed counter (0 when nothing was owed).
  __device__ __forceinline__ uint32_t wait_one(const bfs::PackedWait &w, uint32_t thr, uint32_t known,
                                               uint32_t instance) {
    uint32_t obs = known;
    if (!aborted && thr > 0 && (obs < thr || (kInstr && log))) {
      const uint32_t a = counter_addr(w.w0 & 0xffu);
      obs = uniform(lds_poll(a));
      if (kInstr && st.on) st.polls += 1;
      if (obs < thr) obs = block(a, thr, w.w3 & 0xffffu, instance).observed;
    }
    logit(w.w3 & 0xffffu, instance, thr, thr > 0 ? obs : 0u);
    return obs;
  }

  // A marker / acquire instruction: its waits, then retirement in order.
  __device__ __forceinline__ void nop(kconst<InstrSync> &s, uint32_t instance) {
    for (int j = 0; j < s.n; ++j) {
      const bfs::PackedWait w = C.waits[s.first + j];
      wait_one(w, threshold(w), 0u, instance);
    }
    if (s.update >= 0) {
      retire_all();
      drain_lds();
      add_one(counter_addr((uint32_t)s.update));
    }
  }

  __device__ __forceinline__ void nops(kconst<InstrSync> *list, int n, uint32_t instance) {
    for (int i = 0; i < n; ++i) nop(list[i], instance);
  }

  __device__ __forceinline__ void sync_point() {
    if (kMode == BFS_MODE_BARRIER) {
      retire_all();
      const uint64_t t0 = (kInstr && st.on) ? now_ticks() : 0;
      region_sync(counter_addr((uint32_t)wave), 1);
      if (kInstr && st.on) st.barrier += now_ticks() - t0;
    }
  }
};

// One wait of the innermost instruction in the form evaluated per iteration.
// With r_P the loop register of the producer's loop P, the threshold of Eq. 5
// at an iteration of loop I is
//     thr = [rhat_S > k] * max(run, 0),   run = N * r_P - c,
// and run is carried incrementally (loop-invariant code motion of the wait
// value, Section 6.2): it grows by N whenever r_P is incremented, i.e. per
// iteration of I, M or O according to P, and is never recomputed.  The mask
// reads rhat of loop S: for S = I it becomes "rhat_I > kk" with kk fixed; for
// S = O or M, kk is 0 or "never" per trip of I.  The values are exactly those
// of Eq. 5.
//
// Barrier-free, uninstrumented launches run trips of I in batches of
// consecutive instances; a batch waits for the threshold of its last
// instance, which is the largest of the batch (run and the mask only grow
// with rhat_I), and compares it with `cmp`, the last observed counter value.
struct InnerWait {
  uint32_t addr;       // LDS address of the producer's counter word
  uint32_t dep;        // dependency id (debug log, error word)
  uint32_t bar_thr;    // barrier mode: the static ordinal, 0 when nothing is owed
  uint32_t k;          // the mask is rhat_S > k
  uint32_t kk_lvl;     // 1 / 2: the mask reads rhat of O / M and kk is set per trip; 0: kk is fixed
  uint32_t kk;         // the threshold is 0 while rhat_I <= kk
  int32_t step_i, step_m, step_o;   // N added to run per iteration of I / M / O
  int32_t run;         // N * r_P - c at the current iteration
  int32_t seen;        // last observed counter value (general loop)
  int32_t cmp;         // last observed counter value (batches)
};

// Counter values stay below 2^31; an engine that gave up on a wait marks
// every inner wait as satisfied with this value and finishes without waiting.
constexpr int32_t kSeenAll = 0x7fffffff;
// Instances per batch: 64 lanes move 16 bytes each, four 256-byte tiles.
constexpr uint32_t kBatchMax = 4;

__device__ __forceinline__ InnerWait make_inner(const bfs::PackedWait w, uint32_t cnt_base) {
  InnerWait iw;
  const uint32_t N = w.w1 & 0xffffu, K = w.w1 >> 16, k = w.w2 & 0xffffu, sub = w.w2 >> 16;
  const uint32_t lp = (w.w0 >> 8) & 0xffu, ls = (w.w0 >> 16) & 0xffu, mask = (w.w0 >> 24) & 1u;
  const uint32_t c = N * sub + (N - K);
  iw.addr = cnt_base + 4u * (w.w0 & 0xffu) * (uint32_t)bfs::kMaxWavesPerEngine;
  iw.dep = w.w3 & 0xffffu;
  iw.bar_thr = ((w.w0 >> 25) & 1u) ? (w.w3 >> 16) : 0u;
  iw.k = k;
  iw.kk_lvl = (mask && (ls == 1u || ls == 2u)) ? ls : 0u;
  // fixed kk: no mask, a mask on rhat_I, or a mask on the top level (rhat 1)
  iw.kk = !mask ? 0u : ls == 3u ? k : (1u > k ? 0u : 0xffffffffu);
  iw.step_i = lp == 3u ? (int32_t)N : 0;
  iw.step_m = lp == 2u ? (int32_t)N : 0;
  iw.step_o = lp == 1u ? (int32_t)N : 0;
  iw.run = (int32_t)((lp == 0u ? N : 0u) - c);   // r of the top level is 1, the others start at 0
  iw.seen = 0;
  iw.cmp = 0;
  return iw;
}

// The 32-bit word at a byte offset from base, read through the scalar cache
// with the offset in a scalar register (no 64-bit address arithmetic).
__device__ __forceinline__ uint32_t ldc_at(const int32_t *base, uint32_t byte_off) {
  return (uint32_t)ldc(reinterpret_cast<const int32_t *>(reinterpret_cast<const char *>(base) + byte_off));
}

// kk of a mask on rhat of O or M, at the statement of loop I.
__device__ __forceinline__ void enter_inner(InnerWait &iw, uint32_t h1, uint32_t h2) {
  if (iw.kk_lvl != 0u) iw.kk = ((iw.kk_lvl == 1u ? h1 : h2) > iw.k) ? 0u : 0xffffffffu;
}

// kNW >= 0: the inner instruction has exactly kNW waits and eligible trips of
// I take the short loop (barrier-free, uninstrumented launches only).
// kNW < 0: up to kMaxInnerWaits waits, counted at run time, every trip on
// the general loop.
template <int kRole, int kMode, bool kInstr, int kInflight, int kNW>
__device__ __forceinline__ void run_engine(kconst<Stream3Params> &P, uint32_t cnt_base, float *ring_x,
                                           float *ring_y) {
  constexpr bool kShort = kNW >= 0;
  constexpr int kSlots = kShort ? kNW : kMaxInnerWaits;
  constexpr bool kBF = kMode == BFS_MODE_BARRIER_FREE;
  const int wave = kRole;
  const uint32_t lane = lane_id();
  const int wg = blockIdx.x;
  kconst<EngineCode> &C = P.eng[kRole];
  Engine<kRole, kMode, kInstr, kInflight> E(P, C, cnt_base, wave, wg);
  if (kInstr) {
    if (P.dbg) E.log = P.dbg + (int64_t)gridDim.x * 3 + ((int64_t)wg * 3 + wave) * 4 * P.dbg_cap;
    if (P.stats) {
      E.st.on = true;
      E.st.t_start = now_ticks();
    }
  }
  const uint32_t per_gen = (uint32_t)P.per_gen, n_gen = (uint32_t)P.n_gen;
  const int n_iw = kShort ? kNW : C.inner.n;
  InnerWait iw[kSlots > 0 ? kSlots : 1];
  bool outer_masks = false;   // some wait's mask reads rhat of O or M
#pragma unroll
  for (int j = 0; j < kSlots; ++j)
    if (j < n_iw) {
      iw[j] = make_inner(C.waits[C.inner.first + j], cnt_base);
      outer_masks = outer_masks || iw[j].kk_lvl != 0u;
    }
  {
    // lane 0 adds to the inner instruction's counter, or to its own scratch
    // word when the instruction has no consumer
    const uint32_t scratch = cnt_base + (uint32_t)bfs::kMaxSlots * bfs::kMaxWavesPerEngine * 4u + 256u * (uint32_t)wave;
    E.scratch_v = scratch + 4u * lane;
    const bool counted = C.inner.update >= 0;
    E.own_vaddr = (lane == 0 && counted) ? E.counter_addr((uint32_t)C.inner.update) : E.scratch_v;
    E.one_v = lane == 0 ? 1u : 0u;
  }
  const int64_t *toff = P.trip_off + (int64_t)wg * 4;
  const int64_t tbase = ldc(P.base + wg);
  // per-lane addresses of the rings and of this workgroup's tiles
  const uint32_t xlds = lds_addr(ring_x);                 // LDS byte address of the ring loaded into
  const uint32_t xl = xlds + 4u * lane, yl = lds_addr(ring_y) + 4u * lane;
  const float *xg = P.x + tbase * 64 + lane;
  float *yg = P.y + tbase * 64 + lane;
  // batches: lane l moves bytes [16 l, 16 l + 16) of a block of tiles
  const uint32_t xl4 = lds_addr(ring_x) + 16u * lane, yl4 = lds_addr(ring_y) + 16u * lane;
  const float *xb = P.x + tbase * 64 + 4 * lane;
  float *yb = P.y + tbase * 64 + 4 * lane;
  float addc;   // held in a vector register for the whole run
  asm volatile("v_mov_b32 %0, %1" : "=v"(addc) : "s"(P.addc));
  const uint32_t gen_bytes = 256u * per_gen, ring_bytes = gen_bytes * n_gen;
  const uint32_t kb = min(kBatchMax, per_gen);            // the largest trip one batch holds
  // M iterations run in pairs when the engine has no M-level instruction and
  // no wait whose mask reads rhat of O or M
  const bool pair_ok = kShort && C.n_m_pre == 0 && C.n_m_post == 0 && !outer_masks;

  E.sync_point();                                         // before loop O
  const uint32_t trip_o = (uint32_t)ldc(P.trips + ldc(toff + 1));
  const int64_t off_m = ldc(toff + 2), off_i = ldc(toff + 3);
  uint32_t soff0 = 0;                                     // byte offset of slot ((r_M - 1) % n_gen) * per_gen
  for (uint32_t o = 0; o < trip_o; ++o) {
    E.r1 += 1;
    E.h1 = o + 1;
#pragma unroll
    for (int j = 0; j < kSlots; ++j)
      if (kBF && j < n_iw) iw[j].run += iw[j].step_o;
    E.nops(C.o_pre, C.n_o_pre, E.r1 - 1);
    E.sync_point();                                       // before loop M
    uint32_t trip_m = (uint32_t)ldc(P.trips + off_m + E.r1 - 1);
    if (__builtin_expect(trip_m > P.max_trip_m, 0)) {
      if (kRole == ROLE_LOAD)
        report_input(P.err, 4u, (uint32_t)wg, E.r1 - 1, trip_m, P.max_trip_m, (uint32_t)wave);
      trip_m = P.max_trip_m;
    }
    const int32_t *trip_i_of = P.trips + off_i + E.r2;    // trips of I for this O iteration's M iterations
    // The trips of the next two M iterations are fetched ahead: tq0 for
    // M iteration m + 1, tq1 for m + 2 (indices clamped to the table).
    uint32_t tq0 = trip_m > 0u ? (uint32_t)ldc(trip_i_of) : 0u;
    uint32_t tq1 = trip_m > 1u ? (uint32_t)ldc(trip_i_of + 1) : 0u;
    asm volatile("" ::"s"(tq0), "s"(tq1));   // waited for here, once per O iteration
    uint32_t m = 0;
    while (m < trip_m) {
      if (kShort && pair_ok && m + 1u < trip_m && tq0 - 1u < kb && tq1 - 1u < kb) {
        // Two M iterations whose trips each fit one batch: one wait, one
        // LDS round trip and one counter add for both.
        const uint32_t ta = tq0, tb = tq1;
        tq0 = ldc_at(trip_i_of, 4u * min(m + 2u, trip_m - 1u));
        tq1 = ldc_at(trip_i_of, 4u * min(m + 3u, trip_m - 1u));
        E.r2 += 2;
        E.h2 = m + 2;
        const uint32_t sa = soff0;
        uint32_t sb = soff0 + gen_bytes;
        if (sb == ring_bytes) sb = 0;
        // the largest threshold of the two trips: the second trip's last
        // instance, or the first's while the second's mask is still 0
#pragma unroll
        for (int j = 0; j < kSlots; ++j) {
          const int32_t run_a = iw[j].run + iw[j].step_m + (int32_t)ta * iw[j].step_i;
          const int32_t run_b = run_a + iw[j].step_m + (int32_t)tb * iw[j].step_i;
          iw[j].run = run_b;
          const int32_t thr = tb > iw[j].kk ? run_b : ta > iw[j].kk ? run_a : 0;
          if (thr > iw[j].cmp) {
            int32_t obs = (int32_t)uniform(lds_poll(iw[j].addr));
            if (obs < thr) {
              const WaitResult r = E.block(iw[j].addr, (uint32_t)thr, iw[j].dep, E.r3 + ta + tb - 1u);
              obs = (int32_t)r.observed;
              if (!r.ok) {
#pragma unroll
                for (int jj = 0; jj < kSlots; ++jj) iw[jj].cmp = kSeenAll;
                obs = kSeenAll;
              }
            }
            iw[j].cmp = obs;
          }
          if (kInstr && E.log) {
            // the instance whose threshold the pair waited for: the second
            // trip's last one, or the first trip's last one while the second
            // trip's mask is still 0
            const uint32_t inst = (tb <= iw[j].kk && ta > iw[j].kk) ? E.r3 + ta - 1u : E.r3 + ta + tb - 1u;
            const uint32_t t = thr > 0 ? (uint32_t)thr : 0u;
            E.logit(iw[j].dep, inst, t, t > 0 ? (uint32_t)iw[j].cmp : 0u);
          }
        }
        const int64_t tile_a = (int64_t)E.r3 * 64, tile_b = tile_a + (int64_t)ta * 64;
        const uint32_t kmax = max(ta, tb);
        if (kRole == ROLE_LOAD) {
          if (lane < 16u * ta)
            __builtin_amdgcn_global_load_lds((const void *)(xb + tile_a), (BFS_LDS void *)(uintptr_t)(xlds + sa), 16, 0, 0);
          E.issued_batch(ta);
          if (lane < 16u * tb)
            __builtin_amdgcn_global_load_lds((const void *)(xb + tile_b), (BFS_LDS void *)(uintptr_t)(xlds + sb), 16, 0, 0);
          // the trips have had the first batch to arrive; taking them before
          // the second counter add keeps that add out of the wait
          asm volatile("" ::"s"(tq0), "s"(tq1));
          E.issued_batch(tb);
        } else {
          // both blocks read with the lanes of the longer trip: the extra
          // lanes read slots of the same generations that no engine uses in
          // these M iterations, and their values are dropped
          const uint32_t base = kRole == ROLE_ADD ? xl4 : yl4;
          // (lanes beyond the longer trip leave va and vb undefined: they
          // store and write nothing)
          f32x4 va, vb;
          if (lane < 16u * kmax)
            asm volatile("ds_read_b128 %0, %2\n\tds_read_b128 %1, %3\n\ts_waitcnt lgkmcnt(0)"
                         : "=&v"(va), "=&v"(vb) : "v"(base + sa), "v"(base + sb) : "memory");
          asm volatile("" ::"s"(tq0), "s"(tq1));   // arrived by now (see the single batch)
          if (kRole == ROLE_ADD) {
            if (lane < 16u * ta) {
              va = va + addc;
              asm volatile("ds_write_b128 %0, %1" ::"v"(yl4 + sa), "v"(va) : "memory");
            }
            if (lane < 16u * tb) {
              vb = vb + addc;
              asm volatile("ds_write_b128 %0, %1" ::"v"(yl4 + sb), "v"(vb) : "memory");
            }
          } else {
            if (lane < 16u * ta) __builtin_nontemporal_store(va, (f32x4 *)(yb + tile_a));
            if (lane < 16u * tb) __builtin_nontemporal_store(vb, (f32x4 *)(yb + tile_b));
          }
          E.add_own(ta + tb);
        }
        E.r3 += ta + tb;
        E.h3 = tb;
        soff0 = sb + gen_bytes;
        if (soff0 == ring_bytes) soff0 = 0;
        m += 2;
        asm volatile("" ::"s"(tq0), "s"(tq1));   // taken already (see the end of the loop body)
        continue;
      }
      E.r2 += 1;
      E.h2 = m + 1;
#pragma unroll
      for (int j = 0; j < kSlots; ++j)
        if (kBF && j < n_iw) iw[j].run += iw[j].step_m;
      E.nops(C.m_pre, C.n_m_pre, E.r2 - 1);
      E.sync_point();                                     // before loop I
      const uint32_t trip_i = tq0;
      tq0 = tq1;
      tq1 = ldc_at(trip_i_of, 4u * min(m + 2u, trip_m - 1u));
      if (kShort) {
        // Batches of up to kBatchMax instances within one generation of
        // slots: the tiles of consecutive r_I are adjacent in HBM and their
        // slots adjacent in LDS, so each engine moves a batch as one
        // contiguous block with one 16-byte-per-lane access (lanes from
        // 16 k idle), waits once and adds k to its counter once.  Waiting for
        // the batch's last instance and signalling completions together only
        // delays the engines.
        auto batch = [&](uint32_t k, uint32_t done, uint32_t boff) __attribute__((always_inline)) {
#pragma unroll
          for (int j = 0; j < kSlots; ++j) {
            const int32_t run_last = iw[j].run + (int32_t)k * iw[j].step_i;
            iw[j].run = run_last;
            if (run_last > iw[j].cmp && done + k > iw[j].kk) {
              int32_t obs = (int32_t)uniform(lds_poll(iw[j].addr));
              if (obs < run_last) {
                const WaitResult r = E.block(iw[j].addr, (uint32_t)run_last, iw[j].dep, E.r3 + done + k - 1u);
                obs = (int32_t)r.observed;
                if (!r.ok) {
#pragma unroll
                  for (int jj = 0; jj < kSlots; ++jj) iw[jj].cmp = kSeenAll;
                  obs = kSeenAll;
                }
              }
              iw[j].cmp = obs;
            }
            if (kInstr && E.log) {
              // one entry per batch wait: the batch's last instance
              const uint32_t t = (done + k > iw[j].kk && run_last > 0) ? (uint32_t)run_last : 0u;
              E.logit(iw[j].dep, E.r3 + done + k - 1u, t, t > 0 ? (uint32_t)iw[j].cmp : 0u);
            }
          }
          const int64_t tile = (int64_t)(E.r3 + done) * 64;    // element offset of the batch's first tile
          const bool act = lane < 16u * k;
          if (kRole == ROLE_LOAD) {
            if (act)
              __builtin_amdgcn_global_load_lds((const void *)(xb + tile), (BFS_LDS void *)(uintptr_t)(xlds + boff), 16, 0,
                                               0);
            // the next trip has arrived by now; taking it here keeps its
            // wait ahead of the counter add, which then never holds up the
            // next M iteration
            asm volatile("" ::"s"(tq1));
            E.issued_batch(k);   // batch loads land in issue order
          } else if (kRole == ROLE_ADD) {
            f32x4 v;   // undefined in the idle lanes, which write nothing
            if (act)
              asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(xl4 + boff) : "memory");
            asm volatile("" ::"s"(tq1));   // arrived by now (see the load engine)
            if (act) {
              v = v + addc;
              asm volatile("ds_write_b128 %0, %1" ::"v"(yl4 + boff), "v"(v) : "memory");
            }
            E.add_own(k);   // executed by LDS after the write
          } else {
            if (act) {
              f32x4 v;
              asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(yl4 + boff) : "memory");
              __builtin_nontemporal_store(v, (f32x4 *)(yb + tile));
            }
            asm volatile("" ::"s"(tq1));   // arrived by now (see the load engine)
            E.add_own(k);   // the slots have been read: the stores retire now
          }
        };
        if (__builtin_expect(outer_masks, 0)) {
#pragma unroll
          for (int j = 0; j < kSlots; ++j) enter_inner(iw[j], E.h1, E.h2);
        }
        uint32_t trip_i_v = trip_i;
        if (trip_i - 1u < kb) {
          batch(trip_i, 0u, soff0);                         // the whole trip in one batch
        } else if (trip_i == 0u) {
          asm volatile("" ::"s"(tq1));
        } else {
          if (trip_i > P.max_trip_i) {
            if (kRole == ROLE_LOAD)
              report_input(P.err, 4u, (uint32_t)wg, E.r2 - 1, trip_i, P.max_trip_i, (uint32_t)wave);
            trip_i_v = P.max_trip_i;
          }
          const uint32_t trip_i = trip_i_v;
          // slot = slot0 + (rhat_I - 1) % per_gen: batches never straddle a wrap
          uint32_t done = 0, pos = 0;
          while (done != trip_i) {
            const uint32_t k = min(min(trip_i - done, kBatchMax), per_gen - pos);
            batch(k, done, soff0 + 256u * pos);
            done += k;
            pos += k;
            if (pos == per_gen) pos = 0;
          }
        }
        E.r3 += trip_i_v;
        E.h3 = trip_i_v;
      } else {
        E.flush_batches();
        if (trip_i > P.max_trip_i) {
          if (kRole == ROLE_LOAD)
            report_input(P.err, 4u, (uint32_t)wg, E.r2 - 1, trip_i, P.max_trip_i, (uint32_t)wave);
        }
        const uint32_t trip_i_g = min(trip_i, P.max_trip_i);
#pragma unroll
        for (int j = 0; j < kSlots; ++j)
          if (kBF && j < n_iw) enter_inner(iw[j], E.h1, E.h2);
        uint32_t lo = 0;
        for (uint32_t i = 0; i < trip_i_g; ++i) {
          E.r3 += 1;
          E.h3 = i + 1;
          const uint32_t instance = E.r3 - 1;
#pragma unroll
          for (int j = 0; j < kSlots; ++j) {
            if (j < n_iw) {
              uint32_t thr;
              if (!kBF) {
                thr = iw[j].bar_thr;
              } else {
                iw[j].run += iw[j].step_i;
                thr = (E.h3 > iw[j].kk && iw[j].run > 0) ? (uint32_t)iw[j].run : 0u;
              }
              const uint32_t dep = iw[j].dep;
              if (kInstr && (int)dep == P.fault_dep) thr += (uint32_t)P.fault_delta;
              if (thr > (uint32_t)iw[j].seen || (kInstr && E.log)) {
                uint32_t obs = 0;
                if (!E.aborted && thr > 0) {
                  obs = uniform(lds_poll(iw[j].addr));
                  if (kInstr && E.st.on) E.st.polls += 1;
                  if (obs < thr) {
                    const WaitResult r = E.block(iw[j].addr, thr, dep, instance);
                    obs = r.observed;
                    if (!r.ok) {
#pragma unroll
                      for (int jj = 0; jj < kSlots; ++jj) iw[jj].cmp = kSeenAll;
                    }
                  }
                  iw[j].seen = (int32_t)obs;
                }
                E.logit(dep, instance, thr, obs);
              }
            }
          }
          const uint32_t so = soff0 + 256u * lo;
          if (!E.aborted) {
            if (kRole == ROLE_LOAD) {
              __builtin_amdgcn_global_load_lds((const void *)(xg + (int64_t)instance * 64),
                                               (BFS_LDS void *)(ring_x + so / 4u), 4, 0, 0);
              E.pending = (int)uniform((uint32_t)E.pending + 1u);
              if (E.pending == kInflight) E.retire_oldest_of_full();
            } else if (kRole == ROLE_ADD) {
              float v;
              asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(xl + so) : "memory");
              v = v + addc;
              asm volatile("ds_write_b32 %0, %1" ::"v"(yl + so), "v"(v) : "memory");
              E.add_own(1u);
            } else {
              float v;
              asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(yl + so) : "memory");
              __builtin_nontemporal_store(v, yg + (int64_t)instance * 64);
              E.add_own(1u);
            }
          } else {
            E.retire_all();
            E.add_own(1u);
          }
          lo = (lo + 1 == per_gen) ? 0u : lo + 1;
          if (!kBF) {
            E.sync_point();                               // end of an iteration of I
#pragma unroll
            for (int j = 0; j < kSlots; ++j) iw[j].seen = 0;   // counters were reset
          }
        }
      }
      soff0 += gen_bytes;
      if (soff0 == ring_bytes) soff0 = 0;
      E.nops(C.m_post, C.n_m_post, E.r2 - 1);
      E.sync_point();                                     // end of an iteration of M
      m += 1;
      // Every path has taken the fetched trips by now (a no-op where it
      // already waited for them), so none is still in flight where the
      // paths meet and the next fetch into the same registers need not wait.
      asm volatile("" ::"s"(tq0), "s"(tq1));
    }
    E.nops(C.o_post, C.n_o_post, E.r1 - 1);
    E.sync_point();                                       // end of an iteration of O
  }
  E.retire_all();
  drain_all();
  if (kInstr) {
    if (P.dbg && lane == 0) P.dbg[(int64_t)wg * 3 + wave] = E.nlog;
    if (E.st.on && lane == 0) {
      uint64_t *o = P.stats + ((int64_t)wg * 3 + wave) * 8;
      o[0] = now_ticks() - E.st.t_start;
      o[1] = E.st.blocked;
      o[2] = E.st.n_blocked;
      o[3] = E.st.barrier;
      o[4] = E.st.own_loads;
      o[5] = E.st.polls;
      o[6] = 0;
      o[7] = 0;
    }
  }
}

// The exact count of inner waits selects the short-loop engine.
// Barrier-free launches take the batched loop unless asked for the
// per-instance one (per_instance, uninstrumented) or instrumented without
// log_batched; instrumented launches with log_batched log the batched
// loop's waits (one entry per batch).
template <int kRole, int kMode, bool kInstr, int kInflight>
__device__ __forceinline__ void run_role(kconst<Stream3Params> &P, uint32_t cb, float *rx, float *ry) {
  if constexpr (kMode == BFS_MODE_BARRIER_FREE) {
    const bool batched = kInstr ? P.log_batched != 0 : P.per_instance == 0;
    if (batched) {
      const int n = P.eng[kRole].inner.n;
      if (n == 0) run_engine<kRole, kMode, kInstr, kInflight, 0>(P, cb, rx, ry);
      else if (n == 1) run_engine<kRole, kMode, kInstr, kInflight, 1>(P, cb, rx, ry);
      else run_engine<kRole, kMode, kInstr, kInflight, 2>(P, cb, rx, ry);
      return;
    }
  }
  run_engine<kRole, kMode, kInstr, kInflight, -1>(P, cb, rx, ry);
}

template <int kMode, bool kInstr, int kInflight>
__global__ void __launch_bounds__(192) stream3_kernel(Stream3Params) {
  kconst<Stream3Params> &P = *(kconst<Stream3Params> *)__builtin_amdgcn_kernarg_segment_ptr();
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  uint32_t *cnt = reinterpret_cast<uint32_t *>(lds);
  // counters | 3 x 256 B of per-wave scratch words for the retirement adds | rings
  float *rings = reinterpret_cast<float *>(lds + bfs::kMaxSlots * bfs::kMaxWavesPerEngine * 4 + 768);
  const int ring_floats = P.n_slots * 64;
  for (int i = threadIdx.x; i < bfs::kMaxSlots * bfs::kMaxWavesPerEngine; i += blockDim.x) cnt[i] = 0;
  __syncthreads();
  const uint32_t cb = lds_addr(cnt);
  const int wave = wave_id();
  // Issue priority follows the chain: the load engine, which every other
  // engine waits for, wins arbitration against the add engine, and both
  // against the store engine.
  if (wave == ROLE_LOAD) __builtin_amdgcn_s_setprio(3);
  else if (wave == ROLE_ADD) __builtin_amdgcn_s_setprio(2);
  // run_role(ring read or loaded into, ring written or read from)
  if (wave == ROLE_LOAD) {
    float *r = rings + P.ring_ld * ring_floats;
    run_role<ROLE_LOAD, kMode, kInstr, kInflight>(P, cb, r, r);
  } else if (wave == ROLE_ADD) {
    run_role<ROLE_ADD, kMode, kInstr, kInflight>(P, cb, rings + P.ring_add_src * ring_floats,
                                                 rings + P.ring_add_dst * ring_floats);
  } else {
    float *r = rings + P.ring_st * ring_floats;
    run_role<ROLE_STORE, kMode, kInstr, kInflight>(P, cb, r, r);
  }
}

template <int kMode, bool kInstr>
void launch_variant(const Stream3Params &P, int n_wg, size_t lds, hipStream_t s) {
  if (P.n_slots >= 32) hipLaunchKernelGGL((stream3_kernel<kMode, kInstr, 12>), dim3(n_wg), dim3(192), lds, s, P);
  else hipLaunchKernelGGL((stream3_kernel<kMode, kInstr, 4>), dim3(n_wg), dim3(192), lds, s, P);
}

// --- host: match the plan against the family's loop structure --------------
struct HostEngine {
  std::vector<int> o_pre, m_pre, m_post, o_post;
  int inner = -1;
};

bool collect(const bfs_plan *p, int loop, int e, bool before_child, std::vector<int> &out) {
  out.clear();
  bool seen_loop = false;
  for (int it = p->body_off[loop]; it < p->body_off[loop + 1]; ++it) {
    if (p->body_kind[it] == 1) { seen_loop = true; continue; }
    if (seen_loop == before_child) continue;
    int b = p->body_id[it];
    for (int j = p->block_off[b]; j < p->block_off[b + 1]; ++j) {
      int ins = p->block_instrs[j];
      if (p->instr_engine[ins] != e) continue;
      if (p->instr_opcode[ins] != 0 || (int)out.size() == kMaxNops) return false;
      out.push_back(ins);
    }
  }
  return true;
}

}  // namespace

namespace bfs {

bfs_status launch_stream3(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                          const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream,
                          uint32_t *dbg, int64_t dbg_cap, const bfs_run_opts &o) {
  if (p->n_loops != 4 || p->loop_parent[1] != 0 || p->loop_parent[2] != 1 || p->loop_parent[3] != 2)
    return fail(BFS_E_UNSUPPORTED, "stream3: loops must be top -> O -> M -> I");
  if (p->n_engines != 3 || p->waves_per_engine[0] != 1 || p->waves_per_engine[1] != 1 || p->waves_per_engine[2] != 1)
    return fail(BFS_E_UNSUPPORTED, "stream3: three single-wave engines");
  if (p->tile_elems != 64) return fail(BFS_E_UNSUPPORTED, "stream3: tile_elems must be 64");
  if (!trips || !trip_off || nbufs < 3) return fail(BFS_E_INVALID, "stream3: needs trips and [base, x, y]");
  for (int it = p->body_off[0]; it < p->body_off[1]; ++it)
    if (p->body_kind[it] != 1) return fail(BFS_E_UNSUPPORTED, "stream3: top level must hold only loop O");
  const std::vector<DevWait> dw = device_waits(p);
  Stream3Params P{};
  HostEngine hosts[3];
  const int want_op[3] = {1, 4, 5};
  int n_gen = -1, per_gen = -1;
  int ring_of[4] = {0, 0, 0, 0};      // load dst, add src, add dst, store src
  float addc = 0.f;
  for (int e = 0; e < 3; ++e) {
    HostEngine H;
    if (!collect(p, 1, e, true, H.o_pre) || !collect(p, 1, e, false, H.o_post) || !collect(p, 2, e, true, H.m_pre) ||
        !collect(p, 2, e, false, H.m_post))
      return fail(BFS_E_UNSUPPORTED, "stream3: O and M bodies may hold at most 4 no-op instructions per engine");
    for (int it = p->body_off[3]; it < p->body_off[4]; ++it) {
      if (p->body_kind[it] != 0) return fail(BFS_E_UNSUPPORTED, "stream3: I is innermost");
      int b = p->body_id[it];
      for (int j = p->block_off[b]; j < p->block_off[b + 1]; ++j) {
        int ins = p->block_instrs[j];
        if (p->instr_engine[ins] != e) continue;
        if (H.inner != -1 || p->instr_opcode[ins] != want_op[e])
          return fail(BFS_E_UNSUPPORTED, "stream3: I body must hold load (E0), add (E1), store (E2)");
        H.inner = ins;
        const int32_t *a = &p->instr_args[8 * ins];
        if (a[2] != 2 || a[4] != 3 || (e != 1 && a[6] != 3))
          return fail(BFS_E_UNSUPPORTED, "stream3: slots must be addressed by (r_M, rhat_I), tiles by r_I");
        if (n_gen == -1) { n_gen = a[3]; per_gen = a[5]; }
        if (a[3] != n_gen || a[5] != per_gen) return fail(BFS_E_UNSUPPORTED, "stream3: inconsistent ring geometry");
        if (e == 1) addc = __builtin_bit_cast(float, a[7]);
        if (e == 0) ring_of[0] = a[1];
        if (e == 1) { ring_of[1] = a[0]; ring_of[2] = a[1]; }
        if (e == 2) ring_of[3] = a[0];
      }
    }
    if (H.inner == -1) return fail(BFS_E_UNSUPPORTED, "stream3: every engine needs its instruction in I");
    hosts[e] = H;
    // Resolve each instruction's waits into the launch arguments.
    EngineCode &C = P.eng[e];
    int nw = 0;
    auto fill = [&](int ins, InstrSync &s) -> bool {
      s.first = (int16_t)nw;
      s.n = 0;
      s.update = (int16_t)p->instr_update[ins];
      for (int wi = p->instr_wait_off[ins]; wi < p->instr_wait_off[ins + 1]; ++wi) {
        if (nw == kMaxWaitsPerEngine) return false;
        if (!pack_wait(dw[p->instr_wait_list[wi]], C.waits[nw])) return false;
        ++nw;
        ++s.n;
      }
      return true;
    };
    bool ok = true;
    for (size_t i = 0; i < H.o_pre.size(); ++i) ok &= fill(H.o_pre[i], C.o_pre[i]);
    for (size_t i = 0; i < H.m_pre.size(); ++i) ok &= fill(H.m_pre[i], C.m_pre[i]);
    for (size_t i = 0; i < H.m_post.size(); ++i) ok &= fill(H.m_post[i], C.m_post[i]);
    for (size_t i = 0; i < H.o_post.size(); ++i) ok &= fill(H.o_post[i], C.o_post[i]);
    C.n_o_pre = (int32_t)H.o_pre.size();
    C.n_m_pre = (int32_t)H.m_pre.size();
    C.n_m_post = (int32_t)H.m_post.size();
    C.n_o_post = (int32_t)H.o_post.size();
    ok &= fill(H.inner, C.inner);
    if (!ok || C.inner.n > kMaxInnerWaits)
      return fail(BFS_E_RESOURCE, "stream3: too many waits per engine (16) or per inner instruction (2)");
  }
  if (n_gen < 1 || per_gen < 1 || n_gen * per_gen > 128) return fail(BFS_E_RESOURCE, "stream3: at most 128 ring slots");
  int n_rings = 0;
  for (int i = 0; i < 4; ++i) {
    if (ring_of[i] < 0 || ring_of[i] > 1) return fail(BFS_E_UNSUPPORTED, "stream3: rings 0 and 1 only");
    n_rings = std::max(n_rings, ring_of[i] + 1);
    if (p->ring_slots[ring_of[i]] < n_gen * per_gen)
      return fail(BFS_E_INVALID, "stream3: ring_slots smaller than the addressed slots");
  }
  // Ring-slot reuse the program orders.  A slot of generation
  // (r_M - 1) % n_gen at position (rhat_I - 1) % per_gen is written again
  // per_gen instances later in a long trip of I, and n_gen iterations of M
  // later (r_M counts across O iterations).  For each ring, its first writer
  // must wait for its last reader before the reuse:
  //   I: a dependency between their I instructions at offset <= per_gen
  //      orders reuse inside a trip; without one a trip of I may not exceed
  //      per_gen;
  //   O: a marker of the reader after M -> an acquire of the writer before M
  //      at offset kO: the generations of kO consecutive O iterations must be
  //      distinct, so an M trip may not exceed n_gen / kO;
  //   M: a marker -> acquire pair at M at offset <= n_gen orders reuse inside
  //      an O iteration; with kO = 1 (all reads of the previous O iteration
  //      drained) the M trip is then unbounded.
  // Barrier mode drains every engine at each iteration end: no bound.
  P.max_trip_m = 0xffffffffu;
  P.max_trip_i = 0xffffffffu;
  if (p->mode == BFS_MODE_BARRIER_FREE) {
    const bool in_place = ring_of[0] == ring_of[3];
    const int pairs[2][2] = {{0, in_place ? 2 : 1}, {1, 2}};
    const int n_pairs = in_place ? 1 : 2;
    auto in_list = [](const std::vector<int> &v, int ins) { return std::find(v.begin(), v.end(), ins) != v.end(); };
    // smallest offset of a dependency rd -> wr matching the level, or -1
    auto prot = [&](int rd, int wr, int level) {
      int best = -1;
      for (size_t d = 0; d < p->deps.size() / 3; ++d) {
        if (!p->dep_linear.empty() && p->dep_linear[d]) continue;
        const int prd = p->deps[3 * d], cns = p->deps[3 * d + 1], k = p->deps[3 * d + 2];
        bool ok = false;
        if (level == 3) ok = prd == hosts[rd].inner && cns == hosts[wr].inner && k >= 1 && k <= per_gen;
        else if (level == 2) ok = in_list(hosts[rd].m_post, prd) && in_list(hosts[wr].m_pre, cns) && k >= 1 && k <= n_gen;
        else ok = in_list(hosts[rd].o_post, prd) && in_list(hosts[wr].o_pre, cns) && k >= 1;
        if (ok && (best < 0 || k < best)) best = k;
      }
      return best;
    };
    bool inner_ok = true, m_ok = true;
    int k_o = 1;
    for (int i = 0; i < n_pairs; ++i) {
      const int wr = pairs[i][0], rd = pairs[i][1];
      inner_ok = inner_ok && prot(rd, wr, 3) > 0;
      m_ok = m_ok && prot(rd, wr, 2) > 0;
      const int ko = prot(rd, wr, 1);
      if (ko < 0)
        return fail(BFS_E_UNSUPPORTED, "stream3: ring reuse across O iterations needs a marker -> acquire "
                                       "dependency at O from the ring's last reader to its first writer");
      k_o = std::max(k_o, ko);
    }
    if (!inner_ok) P.max_trip_i = (uint32_t)per_gen;
    if (!(m_ok && k_o == 1)) P.max_trip_m = (uint32_t)(n_gen / k_o);
  }
  P.per_instance = (o.flags & BFS_RUN_PER_INSTANCE) ? 1 : 0;
  P.log_batched = (dbg && (o.flags & BFS_RUN_LOG_BATCHED) && o.fault_dep < 0) ? 1 : 0;
  P.trips = trips;
  P.trip_off = trip_off;
  P.base = static_cast<const int64_t *>(bufs[0]);
  P.x = static_cast<const float *>(bufs[1]);
  P.y = static_cast<float *>(const_cast<void *>(bufs[2]));
  P.dbg = dbg;
  P.dbg_cap = dbg_cap;
  P.err = img->err;
  P.stats = o.dev_stats;
  P.watchdog = o.watchdog_polls;
  P.fault_dep = o.fault_dep;
  P.fault_delta = o.fault_delta;
  P.n_gen = n_gen;
  P.per_gen = per_gen;
  P.n_slots = n_gen * per_gen;
  P.addc = addc;
  P.ring_ld = ring_of[0];
  P.ring_add_src = ring_of[1];
  P.ring_add_dst = ring_of[2];
  P.ring_st = ring_of[3];
  const size_t lds_bytes = (size_t)kMaxSlots * kMaxWavesPerEngine * 4 + 768 + (size_t)n_rings * P.n_slots * 64 * 4;
  const bool instr = dbg || o.dev_stats || o.fault_dep >= 0;
  hipStream_t s = (hipStream_t)stream;
  if (p->mode == BFS_MODE_BARRIER) {
    if (instr) launch_variant<BFS_MODE_BARRIER, true>(P, n_wg, lds_bytes, s);
    else launch_variant<BFS_MODE_BARRIER, false>(P, n_wg, lds_bytes, s);
  } else {
    if (instr) launch_variant<BFS_MODE_BARRIER_FREE, true>(P, n_wg, lds_bytes, s);
    else launch_variant<BFS_MODE_BARRIER_FREE, false>(P, n_wg, lds_bytes, s);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return fail(BFS_E_DEVICE, std::string("stream3 launch: ") + hipGetErrorString(err));
  return BFS_OK;
}

}  // namespace bfs
