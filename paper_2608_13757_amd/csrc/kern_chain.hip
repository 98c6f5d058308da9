// Two-engine chain: a load engine streams 256-element fp32 tiles through an
// LDS ring, a vector engine accumulates a scaled copy of every tile.  One
// wave per engine; the program is a two-level nest A{ B{ ... } }:
//
//   A{ E0: ACQ                                  (no datapath)
//      B{ E0: LOAD  X[n] -> ring[(rhat_B - 1) % R]   (n = r_B - 1 + base[wg])
//         E1: CONS  acc += c * ring[(rhat_B - 1) % R] } }
//   E1: STORE acc -> out[wg]
//
// Dependencies (from the plan, Eq. 5 on the loop registers): LOAD->CONS at
// offset 0, CONS->LOAD at offset R (a slot is refilled only after its tile
// was read, inside one trip of B), CONS->ACQ at offset 1 (case C3 at A: the
// next trip of B starts filling slot 0 again only after the previous trip's
// reads).  The load engine keeps up to four loads in flight (one 16-byte
// direct-to-LDS load per lane moves a tile) and retires them in issue order
// with counted vmcnt waits; the vector engine signals right after its ring
// read returned.  Barrier mode synchronizes both waves before each loop
// statement and at every iteration end, with static ordinals in a region.
//
// Family contract (BFS_KERNEL_CHAIN): loops top -> A -> B; engines of one
// wave each; ACQ (opcode 0, E0) in A before B; LOAD (1, E0) and CONS (2, E1)
// in B, both slotted by rhat_B modulo R = ring_slots[0] (1..8), LOAD tiles
// indexed by r_B; STORE (3, E1) at the top level after A; tile_elems 256.
// Buffers: [0] int64 tile base per workgroup, [1] fp32 input tiles
// [n][256], [2] fp32 output [n_wg][256].
#include <string>

#include "engine_sync.h"

using namespace bfsdev;

namespace {

constexpr int kTileFloats = 256;
constexpr uint32_t kTileBytes = kTileFloats * 4;
constexpr uint32_t kMaxInflight = 4;

struct ChainParams {
  SyncCommon sc;
  InstrWaits acq, load, cons, store;
  const int32_t *trips;
  const int64_t *trip_off;
  const int64_t *base;
  const float *x;
  float *out;
  int32_t ring;
  uint32_t inflight;
  float scale;
};

template <int kMode, bool kInstr>
__global__ void __launch_bounds__(128) chain_kernel(ChainParams P) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  uint32_t *cnt = reinterpret_cast<uint32_t *>(lds);
  unsigned char *ring = lds + kCntBytes;
  for (int i = threadIdx.x; i < bfs::kMaxSlots * bfs::kMaxWavesPerEngine; i += blockDim.x) cnt[i] = 0;
  __syncthreads();

  const int wave = wave_id();
  const uint32_t lane = lane_id();
  const int wg = blockIdx.x;
  Sync<kMode, kInstr> S(P.sc, lds_addr(cnt), wave, wg);
  const int64_t *toff = P.trip_off + (int64_t)wg * 3;
  const uint32_t trip_a = (uint32_t)ldc(P.trips + ldc(toff + 1));
  const int64_t off_b = ldc(toff + 2);
  const int64_t tbase = ldc(P.base + wg);
  const uint32_t R = (uint32_t)P.ring;
  Regs g;

  if (wave == 0) {
    // ------------------------------------------------------------ load engine
    uint32_t pending = 0;                  // loads issued, not yet retired
    auto retire_one = [&]() {              // the oldest load has landed
      wait_vm_dyn((int)pending - 1);
      S.signal(P.load.update, 0);
      pending -= 1;
    };
    auto retire_all = [&]() {
      if (pending > 0) {
        wait_vm<0>();
        for (uint32_t i = 0; i < pending; ++i) S.signal(P.load.update, 0);
        pending = 0;
      }
    };
    const float *src = P.x + tbase * kTileFloats + 4 * lane;
    Site<1> s_acq, s_load;
    S.sync_point(S.word(0, 0));                        // before loop A
    S.enter(s_acq, P.acq, g, 1);
    // the trip of B for the next iteration of A is fetched one iteration ahead
    uint32_t trip_next = trip_a > 0 ? (uint32_t)ldc(P.trips + off_b) : 0u;
    for (uint32_t ia = 0; ia < trip_a; ++ia) {
      g.r1 += 1;
      g.h1 = ia + 1;
      const uint32_t trip_b = trip_next;
      trip_next = (uint32_t)ldc(P.trips + off_b + min(ia + 1u, trip_a - 1u));
      // ACQ: its waits; retired after everything before it
      S.wait(s_acq, P.acq, g, ia + 1, g.r1 - 1, [&] { if (pending > 0) retire_one(); });
      if (P.acq.update >= 0) {
        retire_all();
        S.signal(P.acq.update, 0);
      }
      S.sync_point(S.word(0, 0));                      // before loop B
      S.enter(s_load, P.load, g, 2);
      uint32_t slot = 0;
      for (uint32_t ib = 0; ib < trip_b; ++ib) {
        g.r2 += 1;
        g.h2 = ib + 1;
        S.wait_affine(s_load, P.load, g, ib + 1, g.r2 - 1, [&] { if (pending > 0) retire_one(); });
        if (!S.aborted) {
          __builtin_amdgcn_global_load_lds((const void *)(src + (int64_t)(g.r2 - 1) * kTileFloats),
                                           (BFS_LDS void *)(ring + slot * kTileBytes), 16, 0, 0);
          pending += 1;
          if (pending == P.inflight) retire_one();
        } else {
          S.signal(P.load.update, 0);
        }
        if (kMode == BFS_MODE_BARRIER) {
          retire_all();
          S.sync_point(S.word(0, 0));                  // end of a B iteration
        }
        slot = (slot + 1 == R) ? 0u : slot + 1;
      }
      // The trip's loads are all issued: retire them in order as they land,
      // so the vector engine sees each tile as early as possible (the next
      // ACQ waits for those tiles to be consumed anyway).
      while (pending > 0) retire_one();
      S.sync_point(S.word(0, 0));                      // end of an A iteration
    }
    retire_all();
  } else {
    // ---------------------------------------------------------- vector engine
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    const float c = P.scale;
    Site<1> s_cons, s_store;
    S.sync_point(S.word(1, 0));                        // before loop A
    uint32_t trip_next = trip_a > 0 ? (uint32_t)ldc(P.trips + off_b) : 0u;
    for (uint32_t ia = 0; ia < trip_a; ++ia) {
      g.r1 += 1;
      g.h1 = ia + 1;
      const uint32_t trip_b = trip_next;
      trip_next = (uint32_t)ldc(P.trips + off_b + min(ia + 1u, trip_a - 1u));
      S.sync_point(S.word(1, 0));                      // before loop B
      S.enter(s_cons, P.cons, g, 2);
      uint32_t slot = 0;
      for (uint32_t ib = 0; ib < trip_b; ++ib) {
        g.r2 += 1;
        g.h2 = ib + 1;
        S.wait_affine(s_cons, P.cons, g, ib + 1, g.r2 - 1, [] {});
        if (!S.aborted) {
          const f32x4 v = *(const BFS_LDS f32x4 *)(uintptr_t)(lds_addr(ring) + slot * kTileBytes + 16u * lane);
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[j] = acc[j] + c * v[j];
        }
        // the slot has been read: LDS executes the add after the read
        S.signal(P.cons.update, 0);
        S.sync_point(S.word(1, 0));                    // end of a B iteration (barrier mode)
        slot = (slot + 1 == R) ? 0u : slot + 1;
      }
      S.sync_point(S.word(1, 0));                      // end of an A iteration
    }
    // STORE (top level, after loop A)
    S.enter(s_store, P.store, g, 0);
    S.wait(s_store, P.store, g, 1, 0, [] {});
    if (!S.aborted) __builtin_nontemporal_store(acc, reinterpret_cast<f32x4 *>(P.out + (int64_t)wg * kTileFloats + 4 * lane));
    if (P.store.update >= 0) {
      drain_all();
      S.signal(P.store.update, 0);
    }
  }
  drain_all();
  S.finish(lane);
}

}  // namespace

namespace bfs {

bfs_status launch_chain(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                        const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream, uint32_t *dbg,
                        int64_t dbg_cap, const bfs_run_opts &o) {
  // structure: top{ A{ ACQ(E0); B{ LOAD(E0) CONS(E1) } }; STORE(E1) }
  if (p->n_loops != 3 || p->loop_parent[1] != 0 || p->loop_parent[2] != 1)
    return fail(BFS_E_UNSUPPORTED, "chain: loops must be top -> A -> B");
  if (p->n_engines != 2 || p->waves_per_engine[0] != 1 || p->waves_per_engine[1] != 1)
    return fail(BFS_E_UNSUPPORTED, "chain: two engines of one wave");
  if (p->tile_elems != kTileFloats) return fail(BFS_E_UNSUPPORTED, "chain: tile_elems must be 256");
  int ins_acq = -1, ins_load = -1, ins_cons = -1, ins_store = -1;
  for (size_t i = 0; i < p->instr_engine.size(); ++i) {
    const int op = p->instr_opcode[i], e = p->instr_engine[i], par = p->instr_parent[i];
    if (op == 0 && e == 0 && par == 1 && ins_acq < 0) ins_acq = (int)i;
    else if (op == 1 && e == 0 && par == 2 && ins_load < 0) ins_load = (int)i;
    else if (op == 2 && e == 1 && par == 2 && ins_cons < 0) ins_cons = (int)i;
    else if (op == 3 && e == 1 && par == 0 && ins_store < 0) ins_store = (int)i;
    else return fail(BFS_E_UNSUPPORTED, "chain: unexpected instruction " + std::to_string(i));
  }
  if (ins_acq < 0 || ins_load < 0 || ins_cons < 0 || ins_store < 0)
    return fail(BFS_E_UNSUPPORTED, "chain: needs ACQ, LOAD, CONS and STORE");
  // ACQ precedes loop B in A's body
  auto acq_first = [&]() {
    for (int it = p->body_off[1]; it < p->body_off[2]; ++it) {
      if (p->body_kind[it] == 1) return false;
      for (int j = p->block_off[p->body_id[it]]; j < p->block_off[p->body_id[it] + 1]; ++j)
        if (p->block_instrs[j] == ins_acq) return true;
    }
    return false;
  };
  if (!acq_first()) return fail(BFS_E_UNSUPPORTED, "chain: ACQ must precede loop B");
  const int R = p->ring_slots[0];
  const int32_t *la = &p->instr_args[8 * ins_load];
  const int32_t *ca = &p->instr_args[8 * ins_cons];
  const int32_t *sa = &p->instr_args[8 * ins_store];
  // slot = (rhat_B - 1) % R for both; LOAD reads input buffer 1 at tile r_B
  if (R < 1 || R > 8 || la[0] != 1 || la[1] != 0 || la[2] != -1 || la[4] != 2 || la[5] != R || la[6] != 2 ||
      ca[0] != 0 || ca[1] != 0 || ca[2] != -1 || ca[4] != 2 || ca[5] != R || sa[0] != 0 || sa[1] != 2)
    return fail(BFS_E_UNSUPPORTED, "chain: ring of 1..8 slots indexed by rhat_B, tiles by r_B, one accumulator");
  if (!has_dep(p, ins_load, ins_cons, 0) || !has_dep(p, ins_cons, ins_load, R) || !has_dep(p, ins_cons, ins_acq, 1))
    return fail(BFS_E_UNSUPPORTED, "chain: needs LOAD->CONS(0), CONS->LOAD(ring), CONS->ACQ(1)");
  if (nbufs < 3 || !bufs[0] || !bufs[1] || !bufs[2]) return fail(BFS_E_INVALID, "chain: needs [base, x, out]");
  if (!trips || !trip_off) return fail(BFS_E_INVALID, "chain: needs trip tables");
  const std::vector<DevWait> dw = device_waits(p);
  ChainParams P{};
  if (!fill_waits(p, dw, ins_acq, P.acq) || !fill_waits(p, dw, ins_load, P.load) ||
      !fill_waits(p, dw, ins_cons, P.cons) || !fill_waits(p, dw, ins_store, P.store))
    return fail(BFS_E_RESOURCE, "chain: at most 4 waits per instruction");
  if (!waits_fit({{&P.acq, 1}, {&P.load, 1}, {&P.cons, 1}, {&P.store, 1}}))
    return fail(BFS_E_RESOURCE, "chain: more waits on an instruction than its engine loop takes");
  if (p->mode == BFS_MODE_BARRIER_FREE && (!no_dynamic(P.load) || !no_dynamic(P.cons)))
    return fail(BFS_E_UNSUPPORTED, "chain: a B-loop wait depends on a loop register other than the B loop's");
  P.trips = trips;
  P.trip_off = trip_off;
  P.base = static_cast<const int64_t *>(bufs[0]);
  P.x = static_cast<const float *>(bufs[1]);
  P.out = static_cast<float *>(const_cast<void *>(bufs[2]));
  P.sc = sync_common(img, dbg, dbg_cap, o, 2);
  P.ring = R;
  P.inflight = (uint32_t)R < kMaxInflight ? (uint32_t)R : kMaxInflight;
  P.scale = __builtin_bit_cast(float, ca[7]);
  const size_t lds = kCntBytes + (size_t)R * kTileBytes;
  const bool instr = dbg || o.dev_stats || o.fault_dep >= 0;
  hipStream_t s = (hipStream_t)stream;
  auto go = [&](auto kern) -> bfs_status {
    hipLaunchKernelGGL(kern, dim3(n_wg), dim3(128), lds, s, P);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("chain launch: ") + hipGetErrorString(e));
    return BFS_OK;
  };
  if (p->mode == BFS_MODE_BARRIER)
    return instr ? go(chain_kernel<BFS_MODE_BARRIER, true>) : go(chain_kernel<BFS_MODE_BARRIER, false>);
  return instr ? go(chain_kernel<BFS_MODE_BARRIER_FREE, true>) : go(chain_kernel<BFS_MODE_BARRIER_FREE, false>);
}

}  // namespace bfs
