// AdamW optimizer step (Adam with decoupled weight decay) over fp32
// parameters, with three engines per workgroup over a loop C of parameter
// chunks:
//
//   E0 (1 wave, load)      LOAD: copy one chunk of p, g, m and v from HBM
//                          into a ring slot with direct-to-LDS loads.
//   E1 (W waves, vector)   UPDATE: m' = b1 m + (1 - b1) g,
//                          v' = b2 v + (1 - b2) g^2,
//                          p' = p - lr (c1 m' / (sqrt(c2 v') + eps) + wd p),
//                          with the bias corrections c1 = 1 / (1 - b1^t),
//                          c2 = 1 / (1 - b2^t) of step t; fp32, written in
//                          place into the slot's p, m and v parts.
//   E2 (1 wave, store)     STORE: copy p', m' and v' from the slot to HBM.
//
// Dependencies (from the plan, Eq. 5 on the loop registers): LOAD->UPDATE
// and UPDATE->STORE at offset 0, STORE->LOAD at offset = ring slots (a slot
// is refilled only after its results left): with two slots, offsets {0, 2}.
// Barrier mode synchronizes all waves before the loop and at every iteration
// end.
//
// Layouts.  p, g, m, v fp32 [N] (N a multiple of 4; the last chunk may be
// partial: lanes past N load the last 4 values and store nothing).  A slot
// holds the chunk's p | g | m | v, CH floats each.  Vector wave w updates the 256-float blocks
// w, w + W, ... of the chunk, 4 consecutive floats per lane.
//
// Family contract (BFS_KERNEL_ADAMW): instructions LOAD (E0), UPDATE (E1),
// STORE (E2) in loop C, the only loop below the top level; waves per engine
// 1, W (1, 2 or 4), 1.  LOAD's args hold N, the chunk size CH (256, 512 or
// 1024) and the ring depth; UPDATE's args hold lr, b1, b2, eps, wd (fp32
// bits) and the step t.  Buffers: [0] int64 first chunk per workgroup, [1] p,
// [2] g, [3] m, [4] v (p, m, v updated in place).  Workgroup w runs trip(C)
// chunks from its first chunk.
#include <cmath>
#include <cstring>
#include <string>

#include "engine_sync.h"

using namespace bfsdev;

namespace {

struct AdamParams {
  SyncCommon sc;
  InstrWaits load, upd, store;
  const int64_t *chunk_base;
  float *p;
  const float *g;
  float *m;
  float *v;
  const int32_t *trips;
  const int64_t *trip_off;
  int64_t n;
  int32_t ch, nx, wn;
  float lr, b1, b2, eps, wd, c1, c2;
  uint32_t slot_bytes;
};

template <int kMode, bool kInstr>
__global__ void __launch_bounds__(64 * 6) adamw_kernel(AdamParams P) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  uint32_t *cnt = reinterpret_cast<uint32_t *>(lds);
  unsigned char *ring = lds + kCntBytes;
  for (int i = threadIdx.x; i < bfs::kMaxSlots * bfs::kMaxWavesPerEngine; i += blockDim.x) cnt[i] = 0;
  __syncthreads();

  const int wave = wave_id();
  const uint32_t lane = lane_id();
  const int wg = blockIdx.x;
  Sync<kMode, kInstr> S(P.sc, lds_addr(cnt), wave, wg);
  const int64_t *toff = P.trip_off + (int64_t)wg * 2;
  uint32_t trip = (uint32_t)ldc(P.trips + ldc(toff + 1));
  const int64_t c0 = ldc(P.chunk_base + wg);
  const uint32_t CH = (uint32_t)P.ch, W = (uint32_t)P.wn;
  const int64_t n_chunks = (P.n + CH - 1) / CH;
  // the workgroup's chunks must lie inside the parameter vector
  const int64_t room = c0 >= 0 && c0 <= n_chunks ? n_chunks - c0 : 0;
  if ((int64_t)trip > room) {
    report_input(P.sc.err, 1u, (uint32_t)wg, 0u, trip, (uint32_t)room, (uint32_t)wave);
    trip = (uint32_t)room;
  }
  const uint32_t blocks = CH / 256u;      // 1 KiB blocks per array and chunk
  Regs g;

  if (wave == 0) {
    // ------------------------------------------------------------ load engine
    const uint32_t per_step = 4u * blocks;
    uint32_t pending = 0;
    auto retire_one = [&]() {
      wait_vm_atmost((pending - 1u) * per_step);
      S.signal(P.load.update, 0);
      pending -= 1;
    };
    Site<1> s_load;
    S.sync_point(S.word(0, 0));                      // before loop C
    S.enter(s_load, P.load, g, 1);
    uint32_t slot = 0;
    for (uint32_t it = 0; it < trip; ++it) {
      g.r1 += 1;
      g.h1 = it + 1;
      S.wait_affine(s_load, P.load, g, it + 1, g.r1 - 1, [&] { if (pending > 0) retire_one(); });
      if (!S.aborted) {
        const int64_t e0 = (c0 + it) * (int64_t)CH;     // first parameter of the chunk
        unsigned char *dst = ring + slot * P.slot_bytes;
        const float *src[4] = {P.p, P.g, P.m, P.v};
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          for (uint32_t b = 0; b < blocks; ++b) {
            // lanes past N load the last 4 floats instead (never stored), so
            // that every step issues exactly per_step loads: the counted
            // vmcnt waits that retire a step rely on it
            int64_t e = e0 + 256 * (int64_t)b + 4 * (int64_t)lane;
            e = e < P.n ? e : P.n - 4;
            __builtin_amdgcn_global_load_lds((const void *)(src[a] + e),
                                             (BFS_LDS void *)(dst + (size_t)a * CH * 4u + 1024u * b), 16, 0, 0);
          }
        }
        pending += 1;
        if (pending == (uint32_t)P.nx) retire_one();
      } else {
        S.signal(P.load.update, 0);
      }
      if (kMode == BFS_MODE_BARRIER) {
        while (pending > 0) retire_one();
        S.sync_point(S.word(0, 0));                  // end of a C iteration
      }
      slot = (slot + 1 == (uint32_t)P.nx) ? 0u : slot + 1;
    }
    while (pending > 0) retire_one();
  } else if (wave <= (int)W) {
    // ---------------------------------------------------------- vector engine
    const uint32_t ew = (uint32_t)(wave - 1);
    Site<1> s_upd;
    S.sync_point(S.word(1, ew));                     // before loop C
    S.enter(s_upd, P.upd, g, 1);
    uint32_t slot = 0;
    const float ob1 = 1.0f - P.b1, ob2 = 1.0f - P.b2;
    for (uint32_t it = 0; it < trip; ++it) {
      g.r1 += 1;
      g.h1 = it + 1;
      S.wait_affine(s_upd, P.upd, g, it + 1, g.r1 - 1, [] {});
      if (!S.aborted) {
        const uint32_t base = lds_addr(ring) + slot * P.slot_bytes + 16u * lane;
        for (uint32_t b = ew; b < blocks; b += W) {
          const uint32_t ap = base + 1024u * b, ag = ap + CH * 4u, am = ag + CH * 4u, av = am + CH * 4u;
          f32x4 pv = *(const BFS_LDS f32x4 *)(uintptr_t)ap;
          const f32x4 gv = *(const BFS_LDS f32x4 *)(uintptr_t)ag;
          f32x4 mv = *(const BFS_LDS f32x4 *)(uintptr_t)am;
          f32x4 vv = *(const BFS_LDS f32x4 *)(uintptr_t)av;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float mj = P.b1 * mv[j] + ob1 * gv[j];
            const float vj = P.b2 * vv[j] + ob2 * (gv[j] * gv[j]);
            const float upd = (P.c1 * mj) / (__builtin_sqrtf(P.c2 * vj) + P.eps) + P.wd * pv[j];
            pv[j] = pv[j] - P.lr * upd;
            mv[j] = mj;
            vv[j] = vj;
          }
          *(BFS_LDS f32x4 *)(uintptr_t)ap = pv;
          *(BFS_LDS f32x4 *)(uintptr_t)am = mv;
          *(BFS_LDS f32x4 *)(uintptr_t)av = vv;
        }
      }
      S.signal(P.upd.update, ew);
      S.sync_point(S.word(1, ew));                   // end of a C iteration (barrier mode)
      slot = (slot + 1 == (uint32_t)P.nx) ? 0u : slot + 1;
    }
  } else {
    // ----------------------------------------------------------- store engine
    Site<1> s_store;
    S.sync_point(S.word(2, 0));                      // before loop C
    S.enter(s_store, P.store, g, 1);
    uint32_t slot = 0;
    for (uint32_t it = 0; it < trip; ++it) {
      g.r1 += 1;
      g.h1 = it + 1;
      S.wait_affine(s_store, P.store, g, it + 1, g.r1 - 1, [] {});
      if (!S.aborted) {
        const int64_t e0 = (c0 + it) * (int64_t)CH;
        const uint32_t base = lds_addr(ring) + slot * P.slot_bytes + 16u * lane;
        float *dst[3] = {P.p, P.m, P.v};
        const uint32_t part[3] = {0u, 2u, 3u};
#pragma unroll
        for (int a = 0; a < 3; ++a) {
          for (uint32_t b = 0; b < blocks; ++b) {
            const int64_t e = e0 + 256 * (int64_t)b + 4 * (int64_t)lane;
            const f32x4 d = *(const BFS_LDS f32x4 *)(uintptr_t)(base + part[a] * CH * 4u + 1024u * b);
            if (e < P.n) __builtin_nontemporal_store(d, reinterpret_cast<f32x4 *>(dst[a] + e));
          }
        }
      }
      S.signal(P.store.update, 0);
      S.sync_point(S.word(2, 0));                    // end of a C iteration (barrier mode)
      slot = (slot + 1 == (uint32_t)P.nx) ? 0u : slot + 1;
    }
  }
  drain_all();
  S.finish(lane);
}

}  // namespace

namespace bfs {

bfs_status launch_adamw(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                        const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream, uint32_t *dbg,
                        int64_t dbg_cap, const bfs_run_opts &o) {
  // structure: top{ C{ LOAD(E0) UPDATE(E1) STORE(E2) } }
  if (p->n_loops != 2 || p->loop_parent[1] != 0) return fail(BFS_E_UNSUPPORTED, "adamw: one loop C below the top");
  const int W = p->waves_per_engine[1];
  if (p->n_engines != 3 || p->waves_per_engine[0] != 1 || p->waves_per_engine[2] != 1 || (W != 1 && W != 2 && W != 4))
    return fail(BFS_E_UNSUPPORTED, "adamw: engines of 1, 1/2/4 and 1 waves");
  int ins_load = -1, ins_upd = -1, ins_store = -1;
  for (size_t i = 0; i < p->instr_engine.size(); ++i) {
    const int op = p->instr_opcode[i], e = p->instr_engine[i], par = p->instr_parent[i];
    if (op == 80 && e == 0 && par == 1 && ins_load < 0) ins_load = (int)i;
    else if (op == 81 && e == 1 && par == 1 && ins_upd < 0) ins_upd = (int)i;
    else if (op == 82 && e == 2 && par == 1 && ins_store < 0) ins_store = (int)i;
    else return fail(BFS_E_UNSUPPORTED, "adamw: unexpected instruction " + std::to_string(i));
  }
  if (ins_load < 0 || ins_upd < 0 || ins_store < 0) return fail(BFS_E_UNSUPPORTED, "adamw: needs LOAD, UPDATE and STORE");
  const int32_t *la = &p->instr_args[8 * ins_load];
  const int32_t *ua = &p->instr_args[8 * ins_upd];
  const int64_t N = la[0];
  const int CH = la[1], nx = la[2];
  float hp[5];
  std::memcpy(hp, ua, sizeof(hp));
  const int step = ua[5];
  if (N <= 0 || N % 4 || (CH != 256 && CH != 512 && CH != 1024))
    return fail(BFS_E_UNSUPPORTED, "adamw: N a positive multiple of 4, chunks of 256, 512 or 1024");
  if (nx < 1 || nx > 4) return fail(BFS_E_UNSUPPORTED, "adamw: ring of 1..4 slots");
  if (step < 1 || !(hp[1] >= 0.f && hp[1] < 1.f) || !(hp[2] >= 0.f && hp[2] < 1.f) || !(hp[3] > 0.f))
    return fail(BFS_E_UNSUPPORTED, "adamw: step >= 1, 0 <= b1, b2 < 1, eps > 0");
  if (!has_dep(p, ins_load, ins_upd, 0) || !has_dep(p, ins_upd, ins_store, 0) || !has_dep(p, ins_store, ins_load, nx))
    return fail(BFS_E_UNSUPPORTED, "adamw: needs LOAD->UPDATE(0), UPDATE->STORE(0), STORE->LOAD(ring)");
  if (nbufs < 5 || !bufs[0] || !bufs[1] || !bufs[2] || !bufs[3] || !bufs[4])
    return fail(BFS_E_INVALID, "adamw: needs [chunk base, p, g, m, v]");
  if (!trips || !trip_off) return fail(BFS_E_INVALID, "adamw: needs trip tables");
  const std::vector<DevWait> dw = device_waits(p);
  AdamParams P{};
  if (!fill_waits(p, dw, ins_load, P.load) || !fill_waits(p, dw, ins_upd, P.upd) || !fill_waits(p, dw, ins_store, P.store))
    return fail(BFS_E_RESOURCE, "adamw: at most 4 waits per instruction");
  if (!waits_fit({{&P.load, 1}, {&P.upd, 1}, {&P.store, 1}}))
    return fail(BFS_E_RESOURCE, "adamw: more waits on an instruction than its engine loop takes");
  if (p->mode == BFS_MODE_BARRIER_FREE && (!no_dynamic(P.load) || !no_dynamic(P.upd) || !no_dynamic(P.store)))
    return fail(BFS_E_UNSUPPORTED, "adamw: a chunk-loop wait depends on a loop register other than the chunk loop's");
  P.chunk_base = static_cast<const int64_t *>(bufs[0]);
  P.p = static_cast<float *>(const_cast<void *>(bufs[1]));
  P.g = static_cast<const float *>(bufs[2]);
  P.m = static_cast<float *>(const_cast<void *>(bufs[3]));
  P.v = static_cast<float *>(const_cast<void *>(bufs[4]));
  P.trips = trips;
  P.trip_off = trip_off;
  const int n_waves = W + 2;
  P.sc = sync_common(img, dbg, dbg_cap, o, n_waves);
  P.n = N;
  P.ch = CH;
  P.nx = nx;
  P.wn = W;
  P.lr = hp[0];
  P.b1 = hp[1];
  P.b2 = hp[2];
  P.eps = hp[3];
  P.wd = hp[4];
  // bias corrections of step t, rounded once to fp32
  P.c1 = (float)(1.0 / (1.0 - std::pow((double)hp[1], step)));
  P.c2 = (float)(1.0 / (1.0 - std::pow((double)hp[2], step)));
  P.slot_bytes = 4u * (uint32_t)CH * 4u;
  const size_t lds = kCntBytes + (size_t)nx * P.slot_bytes;
  if (lds > 160 * 1024) return fail(BFS_E_RESOURCE, "adamw: LDS footprint over 160 KiB");
  const bool instr = dbg || o.dev_stats || o.fault_dep >= 0;
  hipStream_t s = (hipStream_t)stream;
  auto go = [&](auto kern) -> bfs_status {
    hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("adamw attribute: ") + hipGetErrorString(e));
    hipLaunchKernelGGL(kern, dim3(n_wg), dim3(64 * n_waves), lds, s, P);
    e = hipGetLastError();
    if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("adamw launch: ") + hipGetErrorString(e));
    return BFS_OK;
  };
  if (p->mode == BFS_MODE_BARRIER)
    return instr ? go(adamw_kernel<BFS_MODE_BARRIER, true>) : go(adamw_kernel<BFS_MODE_BARRIER, false>);
  return instr ? go(adamw_kernel<BFS_MODE_BARRIER_FREE, true>) : go(adamw_kernel<BFS_MODE_BARRIER_FREE, false>);
}

}  // namespace bfs
