// Generic tile-machine interpreter: one wavefront per engine walks its
// projection of the statement tree, maintains the loop registers of
// Section 5.1 (r: entries since the start, rhat: entries in the current
// trip), evaluates every wait before issuing an instruction, executes the
// instruction's datapath and retires it by incrementing its counter.
//
// Family contract (BFS_KERNEL_INTERP): every engine has one wave; buffers are
//   [0] const int64 tile base per workgroup, [1] const fp32 input tiles,
//   [2] fp32 output tiles.
// Opcodes (see the program description): 0 no-op, 1 load tile into a ring
// slot, 2 acc += c * slot, 3 store acc to output tile wg, 4 slot + c into a
// second ring, 5 store a slot to output tile gidx.
#include "bfs_internal.h"
#include "device_sync.h"

using namespace bfsdev;

namespace {

constexpr int kMaxInstrsInterp = 256;

struct InterpParams {
  const int32_t *code;          // int32 x4 words
  const int32_t *code_off;      // [n_engines + 1]
  const bfs::DevWait *waits;    // [n_deps]
  const int32_t *instr_waits;   // CSR [n_instrs + 1]
  const int32_t *waits_by_instr;
  const int32_t *instr_opcode;
  const int32_t *instr_args;    // [n_instrs][8]
  const int32_t *instr_update;  // counter slot or -1
  const int32_t *loop_parent;
  const int32_t *trips;
  const int64_t *trip_off;
  const int64_t *base;
  const float *x;
  float *out;
  uint32_t *dbg;
  int64_t dbg_cap;
  uint32_t *err;
  uint64_t *stats;              // per-wave statistics (null: off)
  uint64_t watchdog;
  int32_t fault_dep, fault_delta;
  int32_t n_loops, n_engines, n_instrs, mode, tile;
  uint32_t fallback_loops;      // bit l: drain barrier at the end of every iteration of loop l
  int32_t ring_off[4];          // float offsets in the ring area
  int32_t acc_off;
  int32_t lds_state_off, lds_exec_off, lds_data_off;   // byte offsets in dynamic LDS
  int32_t lds_snap_off, snap_words;   // per-engine allocation: running counts and snapshots per wave
};

__device__ __forceinline__ int slot_of(const int32_t *a, const uint32_t *r, const uint32_t *rhat) {
  int hi = 0;
  if (a[2] >= 0) hi = (int)((r[a[2]] - 1u) % (uint32_t)a[3]) * a[5];
  int lo = (a[4] >= 0) ? (int)((rhat[a[4]] - 1u) % (uint32_t)a[5]) : 0;
  return hi + lo;
}

__global__ void __launch_bounds__(512) interp_kernel(InterpParams P) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  uint32_t *cnt = reinterpret_cast<uint32_t *>(lds);            // [64 slots][8 waves]
  const int wave = wave_id();
  const uint32_t lane = lane_id();
  const int wg = blockIdx.x;
  uint32_t *st = reinterpret_cast<uint32_t *>(lds + P.lds_state_off) + wave * 3 * bfs::kMaxLoops;
  uint32_t *r = st, *rhat = st + bfs::kMaxLoops, *trip = st + 2 * bfs::kMaxLoops;
  uint32_t *execn = reinterpret_cast<uint32_t *>(lds + P.lds_exec_off) + wave * kMaxInstrsInterp;
  float *data = reinterpret_cast<float *>(lds + P.lds_data_off);
  // per-engine allocation: words 0 .. kMaxEngines - 1 hold the running count
  // of each producer engine's instructions up to this wave's position, then
  // the dependencies' snapshots
  uint32_t *snap = reinterpret_cast<uint32_t *>(lds + P.lds_snap_off) + wave * P.snap_words;

  // Zero counters, state and accumulators.
  for (int i = threadIdx.x; i < bfs::kMaxSlots * bfs::kMaxWavesPerEngine; i += blockDim.x) cnt[i] = 0;
  for (int i = lane; i < 3 * bfs::kMaxLoops; i += 64) st[i] = 0;
  for (int i = lane; i < P.n_instrs; i += 64) execn[i] = 0;
  for (int i = lane; i < P.snap_words; i += 64) snap[i] = 0;
  for (int i = threadIdx.x; i < (P.acc_off + 4 * P.tile); i += blockDim.x) data[i] = 0.f;
  __syncthreads();

  const int e = wave;
  const uint32_t cnt_base = lds_addr(cnt);
  const uint32_t own_words = cnt_base + 4u * (uint32_t)(e * bfs::kMaxWavesPerEngine);
  uint32_t *log_entries = nullptr;
  uint32_t nlog = 0;
  if (P.dbg) {
    const int64_t nw = (int64_t)gridDim.x * P.n_engines;
    log_entries = P.dbg + nw + ((int64_t)wg * P.n_engines + wave) * 4 * P.dbg_cap;
  }
  bool aborted = false;
  WaveStats stt;
  if (P.stats) {
    stt.on = true;
    stt.t_start = now_ticks();
  }
  if (lane == 0) { r[0] = 1; rhat[0] = 1; trip[0] = 1; }
  __builtin_amdgcn_s_waitcnt(0);

  const int32_t *code = P.code + 4 * P.code_off[e];
  int pc = 0;
  const int64_t *toff = P.trip_off + (int64_t)wg * P.n_loops;
  while (true) {
    const int kind = code[4 * pc], a0 = code[4 * pc + 1], a1 = code[4 * pc + 2];
    if (kind == bfs::CODE_HALT) break;
    if (kind == bfs::CODE_LOOP) {
      if (P.mode == BFS_MODE_BARRIER) {
        const uint64_t t0 = stt.on ? now_ticks() : 0;
        region_sync(own_words, 1);
        if (stt.on) stt.barrier += now_ticks() - t0;
      }
      const int l = a0;
      const uint32_t rp = uniform(r[P.loop_parent[l]]);
      const uint32_t t = (uint32_t)P.trips[toff[l] + (int64_t)rp - 1];
      if (lane == 0) { rhat[l] = 0; trip[l] = t; }
      if (t == 0) {
        pc = a1 + 1;
      } else {
        if (lane == 0) { r[l] += 1; rhat[l] = 1; }
        pc += 1;
      }
      __builtin_amdgcn_s_waitcnt(0);
      continue;
    }
    if (kind == bfs::CODE_END) {
      const int l = a0;
      if (P.mode == BFS_MODE_BARRIER) {
        const uint64_t t0 = stt.on ? now_ticks() : 0;
        region_sync(own_words, 1);
        if (stt.on) stt.barrier += now_ticks() - t0;
      } else if ((P.fallback_loops >> l) & 1u) {
        // Section 5.2 fallback: everything issued in this iteration of l has
        // retired on every engine before any engine starts the next one.
        // Every engine walks the same loop tree with the same trip table, so
        // all waves meet the same sequence of barriers.
        drain_all();
        __builtin_amdgcn_s_barrier();
      }
      if (uniform(rhat[l]) < uniform(trip[l])) {
        if (lane == 0) { r[l] += 1; rhat[l] += 1; }
        pc = a1 + 1;
      } else {
        pc += 1;
      }
      __builtin_amdgcn_s_waitcnt(0);
      continue;
    }
    if (kind == bfs::CODE_TRACK) {
      if (lane == 0) snap[a0] += (uint32_t)a1;
      __builtin_amdgcn_s_waitcnt(0);
      pc += 1;
      continue;
    }
    if (kind == bfs::CODE_SNAP) {
      // the producer engine's running count right after the producer's
      // position, kept for the iteration of S it belongs to
      const bfs::DevWait W = P.waits[a0];
      const uint32_t slots = (uint32_t)W.snap_slots;
      const uint32_t idx = slots > 1 ? uniform(r[W.loop_S]) % slots : 0u;
      const uint32_t v = uniform(snap[W.prd_engine]);
      if (lane == 0) snap[W.snap_off + idx] = v;
      __builtin_amdgcn_s_waitcnt(0);
      pc += 1;
      continue;
    }
    // CODE_INSTR
    const int ins = a0;
    const uint32_t inst = uniform(execn[ins]);
    for (int wi = P.instr_waits[ins]; wi < P.instr_waits[ins + 1]; ++wi) {
      const bfs::DevWait W = P.waits[P.waits_by_instr[wi]];
      uint32_t thr;
      if (P.mode == BFS_MODE_BARRIER) {
        thr = W.active ? (uint32_t)W.ordinal : 0u;
      } else if (W.snap_slots > 0) {
        // per-engine: the snapshot of iteration r_S - k (or the latest one),
        // under the mask of Eq. 5
        const uint32_t slots = (uint32_t)W.snap_slots, k = (uint32_t)W.k;
        const uint32_t rS = uniform(r[W.loop_S]), hS = uniform(rhat[W.loop_S]);
        const bool owed = W.linear ? rS > k : (!W.needs_mask || hS > k);
        const uint32_t idx = slots > 1 ? (rS - k) % slots : 0u;
        thr = owed ? uniform(snap[W.snap_off + idx]) : 0u;
      } else {
        thr = eq5(uniform(r[W.loop_P]), uniform(rhat[W.loop_S]), W.k, W.expr_sub, W.N, W.K, W.needs_mask);
      }
      if (W.dep == P.fault_dep) thr += (uint32_t)P.fault_delta;
      WaitResult res{0, true};
      if (!aborted) {
        const uint32_t addr = cnt_base + 4u * (uint32_t)(W.counter * bfs::kMaxWavesPerEngine);
        const uint64_t t0 = stt.on ? now_ticks() : 0;
        res = wait_geq(addr, 1, thr, P.watchdog);
        if (stt.on && thr > 0) {
          const uint64_t dt = now_ticks() - t0;
          stt.blocked += dt;
          stt.n_blocked += 1;
        }
        if (!res.ok) {
          report_deadlock(P.err, (uint32_t)W.dep, (uint32_t)wg, inst, thr, res.observed, (uint32_t)wave);
          aborted = true;
        }
      }
      log_wait(log_entries, P.dbg_cap, nlog, (uint32_t)W.dep, inst, thr, res.observed);
    }
    // Datapath.
    if (!aborted) {
      const int32_t *a = P.instr_args + 8 * ins;
      const int op = P.instr_opcode[ins];
      const int T = P.tile;
      const float c = __int_as_float(a[7]);
      if (op == 1) {          // load
        const int64_t g = P.base[wg] + (int64_t)r[a[6]] - 1;
        float *dst = data + P.ring_off[a[1]] + slot_of(a, r, rhat) * T;
        for (int i = lane; i < T; i += 64) dst[i] = P.x[g * T + i];
      } else if (op == 2) {   // acc += c * slot
        const float *src = data + P.ring_off[a[0]] + slot_of(a, r, rhat) * T;
        float *acc = data + P.acc_off + a[1] * T;
        for (int i = lane; i < T; i += 64) acc[i] = acc[i] + c * src[i];
      } else if (op == 3) {   // store acc
        const float *acc = data + P.acc_off + a[0] * T;
        for (int i = lane; i < T; i += 64) P.out[(int64_t)wg * T + i] = acc[i];
      } else if (op == 4) {   // slot + c
        const int s = slot_of(a, r, rhat);
        const float *src = data + P.ring_off[a[0]] + s * T;
        float *dst = data + P.ring_off[a[1]] + s * T;
        for (int i = lane; i < T; i += 64) dst[i] = src[i] + c;
      } else if (op == 5) {   // store slot
        const int64_t g = P.base[wg] + (int64_t)r[a[6]] - 1;
        const float *src = data + P.ring_off[a[0]] + slot_of(a, r, rhat) * T;
        for (int i = lane; i < T; i += 64) P.out[g * T + i] = src[i];
      }
    }
    // Retire in program order.
    const int upd = P.instr_update[ins];
    if (upd >= 0) retire_all_and_add(cnt_base + 4u * (uint32_t)(upd * bfs::kMaxWavesPerEngine), 1u);
    else drain_all();
    if (lane == 0) execn[ins] = inst + 1;
    __builtin_amdgcn_s_waitcnt(0);
    pc += 1;
  }
  if (P.dbg && lane == 0) P.dbg[(int64_t)wg * P.n_engines + wave] = nlog;
  if (stt.on && lane == 0) {
    uint64_t *o = P.stats + ((int64_t)wg * P.n_engines + wave) * 8;
    o[0] = now_ticks() - stt.t_start;
    o[1] = stt.blocked;
    o[2] = stt.n_blocked;
    o[3] = stt.barrier;
    o[4] = 0;
    o[5] = 0;
    o[6] = 0;
    o[7] = 0;
  }
}

}  // namespace

namespace bfs {

bfs_status launch_interp(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                         const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream,
                         uint32_t *dbg, int64_t dbg_cap, const bfs_run_opts &o) {
  for (int e = 0; e < p->n_engines; ++e)
    if (p->waves_per_engine[e] != 1) return fail(BFS_E_UNSUPPORTED, "interpreter runs one wave per engine");
  if ((int)p->instr_engine.size() > kMaxInstrsInterp) return fail(BFS_E_RESOURCE, "interpreter: > 256 instructions");
  if (!trips || !trip_off) return fail(BFS_E_INVALID, "interpreter needs trip tables");
  if (nbufs < 3) return fail(BFS_E_INVALID, "interpreter needs buffers [base, x, out]");
  InterpParams P{};
  P.code = img->code;
  P.code_off = img->code_off;
  P.waits = img->waits;
  P.instr_waits = img->instr_waits;
  P.waits_by_instr = img->waits_by_instr;
  P.instr_opcode = img->instr_opcode;
  P.instr_args = img->instr_args;
  P.instr_update = img->instr_update;
  P.loop_parent = img->loop_parent;
  P.trips = trips;
  P.trip_off = trip_off;
  P.base = static_cast<const int64_t *>(bufs[0]);
  P.x = static_cast<const float *>(bufs[1]);
  P.out = static_cast<float *>(const_cast<void *>(bufs[2]));
  P.dbg = dbg;
  P.dbg_cap = dbg_cap;
  P.err = img->err;
  P.stats = o.dev_stats;
  P.watchdog = o.watchdog_polls;
  P.fault_dep = o.fault_dep;
  P.fault_delta = o.fault_delta;
  P.n_loops = p->n_loops;
  P.n_engines = p->n_engines;
  P.n_instrs = (int32_t)p->instr_engine.size();
  P.mode = p->mode;
  P.fallback_loops = p->fallback_loops;
  P.tile = p->tile_elems > 0 ? p->tile_elems : 64;
  int off = 0;
  for (int i = 0; i < 4; ++i) {
    P.ring_off[i] = off;
    off += p->ring_slots[i] * P.tile;
  }
  P.acc_off = off;
  off += (p->n_accs > 0 ? p->n_accs : 0) * P.tile;
  const int counters_bytes = kMaxSlots * kMaxWavesPerEngine * 4;
  P.lds_state_off = counters_bytes;
  P.lds_exec_off = P.lds_state_off + p->n_engines * 3 * kMaxLoops * 4;
  P.lds_data_off = P.lds_exec_off + p->n_engines * kMaxInstrsInterp * 4;
  P.snap_words = p->mode == BFS_MODE_BARRIER_FREE && p->alloc == BFS_ALLOC_PER_ENGINE ? p->snap_words : 0;
  P.lds_snap_off = P.lds_data_off + (off + 4 * P.tile) * 4;
  const size_t lds_bytes = (size_t)P.lds_snap_off + (size_t)p->n_engines * P.snap_words * 4;
  if (lds_bytes > 160 * 1024) return fail(BFS_E_RESOURCE, "interpreter: LDS footprint over 160 KiB");
  hipError_t err = hipFuncSetAttribute((const void *)interp_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds_bytes);
  if (err != hipSuccess) return fail(BFS_E_DEVICE, std::string("hipFuncSetAttribute: ") + hipGetErrorString(err));
  hipLaunchKernelGGL(interp_kernel, dim3(n_wg), dim3(64 * p->n_engines), lds_bytes, (hipStream_t)stream, P);
  err = hipGetLastError();
  if (err != hipSuccess) return fail(BFS_E_DEVICE, std::string("interp launch: ") + hipGetErrorString(err));
  return BFS_OK;
}

}  // namespace bfs
