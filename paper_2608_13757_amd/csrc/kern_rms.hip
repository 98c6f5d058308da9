// RMSNorm followed by per-row dynamic FP8 quantization, with three engines
// per workgroup over a software-pipelined row loop R (one row per step):
//
//   E0 (1 wave, load)          LOAD: copy the step's row of X (bf16) from
//                              HBM into an x-ring slot with direct-to-LDS
//                              loads.
//   E1 (W waves, vector)       NORM: wave w takes columns [w H/W, (w+1) H/W)
//                              of the row: its partial sum of squares and
//                              maximum of |x * gamma|, combined over the W
//                              waves through LDS (a fixed summation order, so
//                              every wave gets the same totals); then
//                              y = x * rsqrt(mean(x^2) + eps) * gamma, the
//                              scale s = max|y| / 448 and the OCP E4M3 codes
//                              of y / s (hardware conversion, round to
//                              nearest even; x read a second time from the
//                              slot), written with s into a q-ring slot.  fp32 throughout; y / s is evaluated as
//                              (x * gamma) * (rsqrt(...) * 448 / max|y|), and
//                              max|y| as rsqrt(...) * max|x * gamma| (exact:
//                              rounding is monotone and rsqrt(...) > 0).
//   E2 (1 wave, store)         STORE: copy the step's codes and scale from
//                              the q-ring slot to HBM.
//
// Dependencies (from the plan, Eq. 5 on the loop registers): LOAD->NORM
// (k = 0) and NORM->LOAD (k = x-ring slots) on the x ring, NORM->STORE
// (k = 0) and STORE->NORM (k = q-ring slots) on the q ring: with two slots
// each, loads are double-buffered against stores (offsets {0, 2}).  Barrier
// mode synchronizes all waves before the loop and at every iteration end.
// The vector waves' meeting inside NORM is part of that instruction's
// datapath (a reduction across the engine's own waves), in both modes.
//
// Layouts.  X bf16 [T][H] row-major, gamma bf16 [H], Q uint8 [T][H], S fp32
// [T].  An x slot holds one row as in HBM; lane l of vector wave w owns the
// columns w H/W + 512 c + 8 l .. + 7 for c < H / (512 W) (their gamma
// values stay in registers as fp32), reads them with one 16-byte LDS read
// per c and writes their 8 codes with one 8-byte write.  A q slot holds H
// codes and a 16-byte trailer whose first word is the scale.  After the q
// ring: the reduction area (an arrival counter, then per step parity and
// wave the partial sum of squares and maximum).
//
// Family contract (BFS_KERNEL_RMSNORM): instructions LOAD (E0), NORM (E1),
// STORE (E2) in loop R, the only loop below the top level; waves per engine
// 1, W (1, 2, 4 or 8), 1.  LOAD's args hold T, H and the x-ring depth;
// NORM's args[0] the q-ring depth and args[1] eps (fp32 bits).  H / (512 W)
// is 1, 2 or 4.  Buffers: [0] int64 first row per workgroup, [1] X,
// [2] gamma, [3] Q, [4] S.  Workgroup w runs trip(R) rows from its first
// row.
#include <cstring>
#include <string>
#include <type_traits>

#include "engine_sync.h"

using namespace bfsdev;

namespace {

constexpr int kMaxVecWaves = 8;

struct RmsParams {
  SyncCommon sc;
  InstrWaits load, norm, store;
  const int64_t *row_base;
  const __bf16 *x;
  const __bf16 *gamma;
  uint8_t *q;
  float *s;
  const int32_t *trips;
  const int64_t *trip_off;
  int32_t t, h, wn, nx, nq;               // wn: vector-engine waves
  float eps;
  uint32_t x_slot, q_slot, q_off, red_off;  // bytes: x slot, q slot (codes + trailer), q ring, reduction area
};

// Sum and maximum over the 64 lanes: DPP within rows of 16, then the four
// row results read from lanes 0, 16, 32, 48 (wave-uniform result).
__device__ __forceinline__ float wave_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x124, 0xF, 0xF, false));  // row_ror 4
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x128, 0xF, 0xF, false));  // row_ror 8
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (a + b) + (c + d);
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x124, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x128, 0xF, 0xF, false)));
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return fmaxf(fmaxf(a, b), fmaxf(c, d));
}

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

template <int kMode, bool kInstr, int kC>
__global__ void __launch_bounds__(64 * (kMaxVecWaves + 2)) rms_kernel(RmsParams P) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  uint32_t *cnt = reinterpret_cast<uint32_t *>(lds);
  unsigned char *xring = lds + kCntBytes;
  unsigned char *qring = lds + P.q_off;
  unsigned char *red = lds + P.red_off;
  for (int i = threadIdx.x; i < bfs::kMaxSlots * bfs::kMaxWavesPerEngine; i += blockDim.x) cnt[i] = 0;
  if (threadIdx.x == 0) *reinterpret_cast<uint32_t *>(red) = 0;
  __syncthreads();

  const int wave = wave_id();
  const uint32_t lane = lane_id();
  const int wg = blockIdx.x;
  Sync<kMode, kInstr> S(P.sc, lds_addr(cnt), wave, wg);
  const int64_t *toff = P.trip_off + (int64_t)wg * 2;
  uint32_t trip = (uint32_t)ldc(P.trips + ldc(toff + 1));
  const int64_t row0 = ldc(P.row_base + wg);
  const uint32_t H = (uint32_t)P.h, W = (uint32_t)P.wn;
  // the workgroup's rows must lie inside X
  const int64_t room = row0 >= 0 && row0 <= P.t ? (int64_t)P.t - row0 : 0;
  if ((int64_t)trip > room) {
    report_input(P.sc.err, 1u, (uint32_t)wg, 0u, trip, (uint32_t)room, (uint32_t)wave);
    trip = (uint32_t)room;
  }
  Regs g;

  if (wave == 0) {
    // ------------------------------------------------------------ load engine
    const uint32_t per_step = H / 512u;              // 1 KiB loads per row
    uint32_t pending = 0;                            // issued steps not yet retired
    auto retire_one = [&]() {                        // the oldest step has landed
      wait_vm_atmost((pending - 1u) * per_step);
      S.signal(P.load.update, 0);
      pending -= 1;
    };
    Site<1> s_load;
    S.sync_point(S.word(0, 0));                      // before loop R
    S.enter(s_load, P.load, g, 1);
    uint32_t slot = 0;
    for (uint32_t it = 0; it < trip; ++it) {
      g.r1 += 1;
      g.h1 = it + 1;
      S.wait_affine(s_load, P.load, g, it + 1, g.r1 - 1, [&] { if (pending > 0) retire_one(); });
      if (!S.aborted) {
        const char *src = reinterpret_cast<const char *>(P.x + (size_t)(row0 + it) * H);
        unsigned char *dst = xring + slot * P.x_slot;
        for (uint32_t c = 0; c < per_step; ++c)
          __builtin_amdgcn_global_load_lds((const void *)(src + 1024u * c + 16u * lane), (BFS_LDS void *)(dst + 1024u * c),
                                           16, 0, 0);
        pending += 1;
        if (pending == (uint32_t)P.nx) retire_one();
      } else {
        S.signal(P.load.update, 0);
      }
      if (kMode == BFS_MODE_BARRIER) {
        while (pending > 0) retire_one();
        S.sync_point(S.word(0, 0));                  // end of an R iteration
      }
      slot = (slot + 1 == (uint32_t)P.nx) ? 0u : slot + 1;
    }
    while (pending > 0) retire_one();
  } else if (wave <= (int)W) {
    // ---------------------------------------------------------- vector engine
    const uint32_t ew = (uint32_t)(wave - 1);
    const uint32_t col0 = ew * (H / W) + 8u * lane;  // first column of chunk 0 of this lane
    float gf[kC][8];
#pragma unroll
    for (int c = 0; c < kC; ++c) {
      const u32x4 gv = *reinterpret_cast<const u32x4 *>(P.gamma + col0 + 512u * c);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        gf[c][2 * j] = bf_lo(gv[j]);
        gf[c][2 * j + 1] = bf_hi(gv[j]);
      }
    }
    const uint32_t arrive = lds_addr(red), parts = arrive + 16u;   // parts: [2][kMaxVecWaves] x {ss, m}
    const uint32_t limit = P.sc.watchdog > 0xffffffffull ? 0xffffffffu : (uint32_t)P.sc.watchdog;
    Site<2> s_norm;
    S.sync_point(S.word(1, ew));                     // before loop R
    S.enter(s_norm, P.norm, g, 1);
    uint32_t xs = 0, qs = 0;
    const float inv_h = 1.0f / (float)H;
    for (uint32_t it = 0; it < trip; ++it) {
      g.r1 += 1;
      g.h1 = it + 1;
      S.wait_affine(s_norm, P.norm, g, it + 1, g.r1 - 1, [] {});
      const uint32_t xa = lds_addr(xring) + xs * P.x_slot + 2u * col0;
      float ss = 0.f, mg = 0.f;
      if (!S.aborted) {
#pragma unroll
        for (int c = 0; c < kC; ++c) {
          const u32x4 xv = *(const BFS_LDS u32x4 *)(uintptr_t)(xa + 1024u * c);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float a = bf_lo(xv[j]), b = bf_hi(xv[j]);
            ss = __builtin_fmaf(a, a, ss);
            ss = __builtin_fmaf(b, b, ss);
            mg = fmaxf(mg, fmaxf(__builtin_fabsf(a * gf[c][2 * j]), __builtin_fabsf(b * gf[c][2 * j + 1])));
          }
        }
      }
      // Combine the W waves' partials of this row: each wave writes its
      // pair, then counts itself in; the pair area alternates with the step
      // parity (a wave can be at most one step ahead of a wave that has not
      // read the previous step's pairs, since that step needs its arrival).
      {
        const float ssw = wave_sum(ss), mw = wave_max(mg);
        const uint32_t pa = parts + ((it & 1u) * kMaxVecWaves + ew) * 8u;
        if (lane == 0)
          asm volatile("ds_write_b64 %0, %1" ::"v"(pa), "v"(u32x2{__float_as_uint(ssw), __float_as_uint(mw)}) : "memory");
        lds_add(arrive, 1u);
        const uint32_t target = W * (it + 1u);
        uint32_t polls = 0;
        while (uniform(lds_poll(arrive)) < target) {
          if (++polls > limit) {
            report_deadlock(P.sc.err, 0xffffu, (uint32_t)wg, it, target, uniform(lds_poll(arrive)), (uint32_t)wave);
            S.aborted = 1u;
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        }
      }
      if (!S.aborted) {
        float tot = 0.f, m = 0.f;
        const uint32_t pb = parts + (it & 1u) * kMaxVecWaves * 8u;
        for (uint32_t w = 0; w < W; ++w) {
          const u32x2 v = *(const BFS_LDS u32x2 *)(uintptr_t)(pb + 8u * w);
          tot += __uint_as_float(v.x);
          m = fmaxf(m, __uint_as_float(v.y));
        }
        const float rinv = __builtin_amdgcn_rsqf(tot * inv_h + P.eps);
        const float amax = m > 0.f ? rinv * m : 0.f;   // a zero row keeps scale 1 even with eps = 0
        const float inv = amax > 0.f ? 448.0f / amax : 0.f;
        const float scale = amax > 0.f ? amax / 448.0f : 1.0f;
        const float f = rinv * inv;
        const uint32_t qa = lds_addr(qring) + qs * P.q_slot + col0;
        // second pass: x read again from the slot (registers stay below 64,
        // so three 6-wave workgroups fit on a CU)
#pragma unroll
        for (int c = 0; c < kC; ++c) {
          const u32x4 xv = *(const BFS_LDS u32x4 *)(uintptr_t)(xa + 1024u * c);
          float t[8];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            t[2 * j] = (bf_lo(xv[j]) * gf[c][2 * j]) * f;
            t[2 * j + 1] = (bf_hi(xv[j]) * gf[c][2 * j + 1]) * f;
          }
          int w0 = __builtin_amdgcn_cvt_pk_fp8_f32(t[0], t[1], 0, false);
          w0 = __builtin_amdgcn_cvt_pk_fp8_f32(t[2], t[3], w0, true);
          int w1 = __builtin_amdgcn_cvt_pk_fp8_f32(t[4], t[5], 0, false);
          w1 = __builtin_amdgcn_cvt_pk_fp8_f32(t[6], t[7], w1, true);
          *(BFS_LDS u32x2 *)(uintptr_t)(qa + 512u * c) = u32x2{(uint32_t)w0, (uint32_t)w1};
        }
        if (ew == 0 && lane == 0) *(BFS_LDS float *)(uintptr_t)(lds_addr(qring) + qs * P.q_slot + H) = scale;
      }
      S.signal(P.norm.update, ew);
      S.sync_point(S.word(1, ew));                   // end of an R iteration (barrier mode)
      xs = (xs + 1 == (uint32_t)P.nx) ? 0u : xs + 1;
      qs = (qs + 1 == (uint32_t)P.nq) ? 0u : qs + 1;
    }
  } else {
    // ----------------------------------------------------------- store engine
    Site<1> s_store;
    S.sync_point(S.word(2, 0));                      // before loop R
    S.enter(s_store, P.store, g, 1);
    uint32_t qs = 0;
    for (uint32_t it = 0; it < trip; ++it) {
      g.r1 += 1;
      g.h1 = it + 1;
      S.wait_affine(s_store, P.store, g, it + 1, g.r1 - 1, [] {});
      if (!S.aborted) {
        const int64_t row = row0 + it;
        const uint32_t qa = lds_addr(qring) + qs * P.q_slot;
        for (uint32_t c = 0; c < H / 1024u; ++c) {
          const u32x4 d = *(const BFS_LDS u32x4 *)(uintptr_t)(qa + 1024u * c + 16u * lane);
          __builtin_nontemporal_store(d, reinterpret_cast<u32x4 *>(P.q + (size_t)row * H + 1024u * c + 16u * lane));
        }
        const float sc = *(const BFS_LDS float *)(uintptr_t)(qa + H);
        if (lane == 0) P.s[row] = sc;
      }
      S.signal(P.store.update, 0);
      S.sync_point(S.word(2, 0));                    // end of an R iteration (barrier mode)
      qs = (qs + 1 == (uint32_t)P.nq) ? 0u : qs + 1;
    }
  }
  drain_all();
  S.finish(lane, S.st.t_start);                      // statistics: the wave's start time
}

}  // namespace

namespace bfs {

bfs_status launch_rms(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs, const int32_t *trips,
                      const int64_t *trip_off, int32_t n_wg, void *stream, uint32_t *dbg, int64_t dbg_cap,
                      const bfs_run_opts &o) {
  // structure: top{ R{ LOAD(E0) NORM(E1) STORE(E2) } }
  if (p->n_loops != 2 || p->loop_parent[1] != 0) return fail(BFS_E_UNSUPPORTED, "rmsnorm: one loop R below the top");
  const int W = p->waves_per_engine[1];
  if (p->n_engines != 3 || p->waves_per_engine[0] != 1 || p->waves_per_engine[2] != 1 ||
      (W != 1 && W != 2 && W != 4 && W != 8))
    return fail(BFS_E_UNSUPPORTED, "rmsnorm: engines of 1, 1/2/4/8 and 1 waves");
  int ins_load = -1, ins_norm = -1, ins_store = -1;
  for (size_t i = 0; i < p->instr_engine.size(); ++i) {
    const int op = p->instr_opcode[i], e = p->instr_engine[i], par = p->instr_parent[i];
    if (op == 64 && e == 0 && par == 1 && ins_load < 0) ins_load = (int)i;
    else if (op == 65 && e == 1 && par == 1 && ins_norm < 0) ins_norm = (int)i;
    else if (op == 66 && e == 2 && par == 1 && ins_store < 0) ins_store = (int)i;
    else return fail(BFS_E_UNSUPPORTED, "rmsnorm: unexpected instruction " + std::to_string(i));
  }
  if (ins_load < 0 || ins_norm < 0 || ins_store < 0) return fail(BFS_E_UNSUPPORTED, "rmsnorm: needs LOAD, NORM and STORE");
  const int32_t *la = &p->instr_args[8 * ins_load];
  const int T = la[0], H = la[1], nx = la[2];
  const int nq = p->instr_args[8 * ins_norm];
  float eps;
  std::memcpy(&eps, &p->instr_args[8 * ins_norm + 1], 4);
  if (T <= 0 || H <= 0 || H % 1024 || H > 8192) return fail(BFS_E_UNSUPPORTED, "rmsnorm: T > 0, H a multiple of 1024 up to 8192");
  const int kc = H / (512 * W);
  if (H % (512 * W) || (kc != 1 && kc != 2 && kc != 4))
    return fail(BFS_E_UNSUPPORTED, "rmsnorm: H / (512 x vector waves) must be 1, 2 or 4");
  if (nx < 1 || nx > 4 || nq < 1 || nq > 4 || !(eps >= 0.f))
    return fail(BFS_E_UNSUPPORTED, "rmsnorm: rings of 1..4 slots, eps >= 0");
  // the ring dependencies keep a slot from being refilled before it is read
  if (!has_dep(p, ins_load, ins_norm, 0) || !has_dep(p, ins_norm, ins_store, 0) ||
      !has_dep(p, ins_norm, ins_load, nx) || !has_dep(p, ins_store, ins_norm, nq))
    return fail(BFS_E_UNSUPPORTED, "rmsnorm: needs LOAD->NORM(0), NORM->STORE(0), NORM->LOAD(x ring), STORE->NORM(q ring)");
  if (nbufs < 5 || !bufs[0] || !bufs[1] || !bufs[2] || !bufs[3] || !bufs[4])
    return fail(BFS_E_INVALID, "rmsnorm: needs [row base, X, gamma, Q, S]");
  if (!trips || !trip_off) return fail(BFS_E_INVALID, "rmsnorm: needs trip tables");
  const std::vector<DevWait> dw = device_waits(p);
  RmsParams P{};
  if (!fill_waits(p, dw, ins_load, P.load) || !fill_waits(p, dw, ins_norm, P.norm) ||
      !fill_waits(p, dw, ins_store, P.store))
    return fail(BFS_E_RESOURCE, "rmsnorm: at most 4 waits per instruction");
  if (!waits_fit({{&P.load, 1}, {&P.norm, 2}, {&P.store, 1}}))
    return fail(BFS_E_RESOURCE, "rmsnorm: more waits on an instruction than its engine loop takes");
  if (p->mode == BFS_MODE_BARRIER_FREE && (!no_dynamic(P.load) || !no_dynamic(P.norm) || !no_dynamic(P.store)))
    return fail(BFS_E_UNSUPPORTED, "rmsnorm: a row-loop wait depends on a loop register other than the row loop's");
  P.row_base = static_cast<const int64_t *>(bufs[0]);
  P.x = static_cast<const __bf16 *>(bufs[1]);
  P.gamma = static_cast<const __bf16 *>(bufs[2]);
  P.q = static_cast<uint8_t *>(const_cast<void *>(bufs[3]));
  P.s = static_cast<float *>(const_cast<void *>(bufs[4]));
  P.trips = trips;
  P.trip_off = trip_off;
  const int n_waves = W + 2;
  P.sc = sync_common(img, dbg, dbg_cap, o, n_waves);
  P.t = T;
  P.h = H;
  P.wn = W;
  P.nx = nx;
  P.nq = nq;
  P.eps = eps;
  P.x_slot = (uint32_t)H * 2u;
  P.q_slot = (uint32_t)H + 16u;
  P.q_off = kCntBytes + (uint32_t)nx * P.x_slot;
  P.red_off = P.q_off + (uint32_t)nq * P.q_slot;
  const size_t lds = (size_t)P.red_off + 16 + 2 * kMaxVecWaves * 8;
  if (lds > 160 * 1024) return fail(BFS_E_RESOURCE, "rmsnorm: LDS footprint over 160 KiB");
  const bool instr = dbg || o.dev_stats || o.fault_dep >= 0;
  hipStream_t s = (hipStream_t)stream;
  auto go = [&](auto kern) -> bfs_status {
    hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("rmsnorm attribute: ") + hipGetErrorString(e));
    hipLaunchKernelGGL(kern, dim3(n_wg), dim3(64 * n_waves), lds, s, P);
    e = hipGetLastError();
    if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("rmsnorm launch: ") + hipGetErrorString(e));
    return BFS_OK;
  };
  auto pick = [&](auto mode_tag, auto instr_tag) -> bfs_status {
    constexpr int M = decltype(mode_tag)::value;
    constexpr bool I = decltype(instr_tag)::value;
    if (kc == 1) return go(rms_kernel<M, I, 1>);
    if (kc == 2) return go(rms_kernel<M, I, 2>);
    return go(rms_kernel<M, I, 4>);
  };
  using BF = std::integral_constant<int, BFS_MODE_BARRIER_FREE>;
  using BA = std::integral_constant<int, BFS_MODE_BARRIER>;
  using On = std::true_type;
  using Off = std::false_type;
  if (p->mode == BFS_MODE_BARRIER) return instr ? pick(BA{}, On{}) : pick(BA{}, Off{});
  return instr ? pick(BF{}, On{}) : pick(BF{}, Off{});
}

}  // namespace bfs
