// bf16 GEMM + bias + GELU with three engines per workgroup, one 256 x 256
// output tile per workgroup:
//
//   E0 (2 waves, load)      BIAS: stage the tile's 256 bias values in LDS;
//                           LOAD: copy the A rows and B columns of one 32-wide
//                           K step from HBM into a ring slot with
//                           direct-to-LDS loads (A by wave 0, B by wave 1).
//   E1 (8 waves, MFMA)      MMA: 2 x 8 v_mfma_f32_32x32x16_bf16 per K step on
//                           a 128 x 64 sub-tile per wave, fp32 accumulators;
//                           SPILL: bias + GELU of one 32 x 32 accumulator
//                           block in registers, packed to bf16 into an
//                           epilogue ring slot.
//   E2 (2 waves, epilogue)  EPI: read a chunk from the epilogue ring and
//                           store it to HBM with 16-byte row segments.
//
// Dependencies (from the plan, Eq. 5 on the engines' loop registers):
// LOAD->MMA (k = 0) and MMA->LOAD (k = ring slots) on the K ring, SPILL->EPI
// (k = 0) and EPI->SPILL (k = epilogue slots) on the epilogue ring,
// BIAS->SPILL at the top level.  Every engine wave keeps its own counter word;
// a wait requires all waves of the producer engine.  Barrier mode
// synchronizes all waves before each loop statement and at every iteration
// end, with static ordinals inside a region.
//
// LDS (bytes): counters 2048 | K ring slots of 32 KiB (A 256 x 32 bf16, then
// B 256 x 32 bf16; each row 64 B in four 16-byte chunks stored at chunk
// c ^ ((row / 4) % 4), which makes the MFMA fragment reads conflict-free) |
// bias 1 KiB.  The epilogue slots (1, 2, 4 or 8 of 16 KiB each: 8 blocks of
// 32 x 32 bf16, row-major; chunk c in slot c % slots) reuse the memory of
// the K ring once the K loop is over; the program's MMA->SPILL dependency
// orders every spill after the last K step of every MFMA wave.  With four
// or eight slots the spills of a tile rarely or never wait for the stores.
//
// MFMA operand order: the first operand is the B^T fragment and the second
// the A fragment, so lane l of a 32 x 32 block holds output row (l % 32) and
// columns 8 * (i / 4) + 4 * (l / 32) + i % 4 for accumulator element i: four
// runs of four consecutive columns, written as 8-byte bf16 quads.
//
// GELU uses the exact-erf definition x * Phi(x), with erf evaluated by
// Abramowitz & Stegun formula 7.1.26 (absolute error below 1.5e-7).
//
// Family contract (BFS_KERNEL_GEMM): instructions BIAS (E0, top level),
// LOAD (E0) and MMA (E1) in loop K, SPILL (E1) and EPI (E2) in loop C;
// waves per engine 2, 8, 2.  LOAD's args hold M, N, K and the ring depth;
// SPILL's args[0] the epilogue ring depth.  M and N multiples of 256, K a
// multiple of 32.  Buffers: [0] A bf16 [M][K], [1] B^T bf16 [N][K],
// [2] bias fp32 [N], [3] C bf16 [M][N].  Trip tables: loop K runs K / 32
// steps, loop C 8 chunks.
#include <string>
#include <type_traits>

#include "engine_sync.h"

using namespace bfsdev;

namespace {

constexpr int kTile = 256, kBK = 32;
constexpr int kLoadW = 2, kMmaW = 8, kEpiW = 2, kWaves = 12;
constexpr uint32_t kSlotBytes = 2 * kTile * kBK * 2;     // A + B of one K step
constexpr uint32_t kESlotBytes = kMmaW * 32 * 32 * 2;     // 8 bf16 blocks
constexpr int kMaxSteps = 128;                            // K steps of the K-unrolled program

struct GemmParams {
  SyncCommon sc;
  InstrWaits bias, load, mma, spill, epi;
  const __bf16 *a;
  const __bf16 *bt;
  const float *bias_v;
  __bf16 *c;
  const int32_t *trips;
  const int64_t *trip_off;
  int32_t m, n, k;
  int32_t ring, e_ring;
  int32_t tiles_m, tiles_n;
  int32_t xcd_map;          // 1: group tiles per XCD
  int32_t n_loops;          // 3 (top, K, C) or 2 (top, C: the K-unrolled program)
  // K-unrolled program: counter slots of the top-level LOAD and MMA
  // instructions, and the dependency id of each step's wait (debug log)
  int32_t c_load, c_mma;
  uint16_t dep_mma[kMaxSteps], dep_load[kMaxSteps];
};

__device__ __forceinline__ float gelu_erf(float x) {
  const float z = x * 0.70710678118654752f;
  const float a = __builtin_fabsf(z);
  const float t = __builtin_amdgcn_rcpf(1.0f + 0.3275911f * a);
  const float poly =
      t * (0.254829592f + t * (-0.284496736f + t * (1.421413741f + t * (-1.453152027f + t * 1.061405429f))));
  const float erf_a = 1.0f - poly * __expf(-a * a);
  const float erf_z = __builtin_copysignf(erf_a, z);
  return 0.5f * x * (1.0f + erf_z);
}

__device__ __forceinline__ uint32_t swz(uint32_t row, uint32_t chunk) {
  return row * 64u + ((chunk ^ ((row >> 2) & 3u)) << 4);
}

// kUnroll: K steps per copy of the load and MFMA loop bodies (the trip of
// loop K is static, so an unrolled body sees its thresholds as fixed offsets
// of one value per copy); a remainder of trip_k % kUnroll steps runs singly.
// kSteps > 0: the K-unrolled program (no K loop; kSteps steps in straight
// line at the top level): MMA of step s waits for s + 2 retirements of the
// load engine's top-level counter (BIAS and LOADs 0 .. s), LOAD of step s
// for s - ring + 1 of the MFMA engine's (MMAs 0 .. s - ring), both static
// immediates that the launcher checks against the plan.
template <int kMode, bool kInstr, int kUnroll, int kSteps>
__global__ void __launch_bounds__(768) gemm_kernel(GemmParams P) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  uint32_t *cnt = reinterpret_cast<uint32_t *>(lds);
  unsigned char *ring = lds + kCntBytes;
  unsigned char *ering = ring;                       // reused after the K loop
  float *bias_l = reinterpret_cast<float *>(ring + (size_t)P.ring * kSlotBytes);
  for (int i = threadIdx.x; i < bfs::kMaxSlots * bfs::kMaxWavesPerEngine; i += blockDim.x) cnt[i] = 0;
  __syncthreads();

  const int wave = wave_id();
  const uint32_t lane = lane_id();
  const int wg = blockIdx.x;
  // tile of this workgroup
  int tm, tn;
  if (P.xcd_map) {
    const int xcd = wg & 7, local = wg >> 3;
    const int br = P.tiles_m / 4, bc = P.tiles_n / 2;
    tm = (xcd >> 1) * br + local / bc;
    tn = (xcd & 1) * bc + local % bc;
  } else {
    tm = wg / P.tiles_n;
    tn = wg % P.tiles_n;
  }
  const int m0 = tm * kTile, n0 = tn * kTile;

  Sync<kMode, kInstr> S(P.sc, lds_addr(cnt), wave, wg);
  uint64_t k_end = 0;                      // statistics: end of the K loop
  constexpr bool kFlat = kSteps > 0;
  constexpr uint32_t LC = kFlat ? 1u : 2u;          // loop id of C
  const int64_t *toff = P.trip_off + (int64_t)wg * P.n_loops;
  uint32_t trip_k = kFlat ? (uint32_t)kSteps : (uint32_t)ldc(P.trips + ldc(toff + 1));
  uint32_t trip_c = (uint32_t)ldc(P.trips + ldc(toff + LC));
  if (trip_k > (uint32_t)(P.k / kBK) || trip_c > 8u) {
    report_input(P.sc.err, 2u, (uint32_t)wg, 0u, trip_k, trip_c, (uint32_t)wave);
    trip_k = min(trip_k, (uint32_t)(P.k / kBK));
    trip_c = min(trip_c, 8u);
  }
  Regs g;
  // loop C's registers: r2, h2 below K, or r1, h1 without the K loop
  auto c_iter = [&](uint32_t it) __attribute__((always_inline)) {
    if (kFlat) {
      g.r1 += 1;
      g.h1 = it + 1;
    } else {
      g.r2 += 1;
      g.h2 = it + 1;
    }
  };
  auto c_r = [&]() __attribute__((always_inline)) { return kFlat ? g.r1 : g.r2; };
  const uint32_t ring_base = lds_addr(ring), ering_base = lds_addr(ering);

  if (wave < kLoadW) {
    // ------------------------------------------------------------ load engine
    const uint32_t ew = (uint32_t)wave;
    int pending = 0;                         // outstanding LOAD groups (16 loads each)
    auto retire_one = [&]() {                // the oldest group has landed
      if (pending == 3) wait_vm<32>();
      else if (pending == 2) wait_vm<16>();
      else wait_vm<0>();
      S.signal(P.load.update, ew);
      pending -= 1;
    };
    auto retire_all = [&]() {
      if (pending > 0) {
        wait_vm<0>();
        for (int i = 0; i < pending; ++i) S.signal(P.load.update, ew);
        pending = 0;
      }
    };
    Site<1> s_bias, s_load;
    // BIAS (top level)
    S.enter(s_bias, P.bias, g, 0);
    S.wait(s_bias, P.bias, g, 1, 0, [] {});
    if (wave == 0 && !S.aborted)
      __builtin_amdgcn_global_load_lds((const void *)(P.bias_v + n0 + 4 * lane), (BFS_LDS void *)bias_l, 16, 0, 0);
    wait_vm<0>();
    S.signal(P.bias.update, ew);
    if (!kFlat) S.sync_point(S.word(0, ew));                // before loop K
    // per-lane source rows: lane l covers row 16 j + l / 4, logical chunk
    // (l % 4) ^ ((l / 16) % 4), so its 16 bytes land at the swizzled place.
    const uint32_t r_in = lane >> 2, chunk = (lane & 3u) ^ ((lane >> 4) & 3u);
    if (!kFlat) S.enter(s_load, P.load, g, 1);
    uint32_t seen_mma = 0;
    // A wave-uniform base that advances one K step per iteration plus fixed
    // 32-bit per-lane byte offsets (one per 16-row group): the loads take the
    // scalar-base address form and need no vector address arithmetic, which
    // would compete for issue with the MFMA waves sharing this SIMD.
    const char *sbase = reinterpret_cast<const char *>(wave == 0 ? P.a + (size_t)m0 * P.k : P.bt + (size_t)n0 * P.k);
    uint32_t voff[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) voff[j] = ((16u * j + r_in) * (uint32_t)P.k + 8u * chunk) * 2u;
    uint32_t slot = 0;
    auto load_step = [&](uint32_t it) __attribute__((always_inline)) {
      if (kFlat) {
        if (it >= (uint32_t)P.ring)
          S.wait_fixed((uint32_t)P.c_mma, kMmaW, it - (uint32_t)P.ring + 1u, P.dep_load[it], 0u, seen_mma,
                       [&] { if (pending > 0) retire_one(); });
      } else {
        g.r1 += 1;
        g.h1 = it + 1;
        S.wait_affine(s_load, P.load, g, it + 1, g.r1 - 1, [&] { if (pending > 0) retire_one(); });
      }
      if (!S.aborted) {
        unsigned char *dst = ring + slot * kSlotBytes + (wave == 0 ? 0u : kSlotBytes / 2);
        const char *sb = sbase + (size_t)it * (kBK * 2);
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          asm volatile("" : "+v"(voff[j]));   // keep the offset a 32-bit value at its use
          __builtin_amdgcn_global_load_lds((const void *)(sb + voff[j]), (BFS_LDS void *)(dst + j * 1024), 16, 0, 0);
        }
        pending += 1;
        if (pending == 3) retire_one();
      } else {
        S.signal(P.load.update, ew);
      }
      if (kMode == BFS_MODE_BARRIER && !kFlat) {
        retire_all();
        S.sync_point(S.word(0, ew));                        // end of a K iteration
      }
      slot = (slot + 1 == (uint32_t)P.ring) ? 0u : slot + 1;
    };
    if constexpr (kFlat) {
#pragma unroll
      for (int st = 0; st < kSteps; ++st) load_step((uint32_t)st);
    } else {
      uint32_t it = 0;
      for (; it + kUnroll <= trip_k; it += kUnroll) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) load_step(it + u);
      }
      for (; it < trip_k; ++it) load_step(it);
    }
    retire_all();
    k_end = S.elapsed();
    S.sync_point(S.word(0, ew));                            // before loop C
    for (uint32_t it = 0; it < trip_c; ++it) {
      c_iter(it);
      S.sync_point(S.word(0, ew));                          // end of a C iteration
    }
  } else if (wave < kLoadW + kMmaW) {
    // ------------------------------------------------------------ MFMA engine
    const uint32_t ew = (uint32_t)(wave - kLoadW);
    const uint32_t wm = ew >> 2, wn = ew & 3u;
    f32x16 acc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = f32x16{};
    Site<1> s_mma;
    Site<3> s_spill;
    if (!kFlat) {
      S.sync_point(S.word(1, ew));                          // before loop K
      S.enter(s_mma, P.mma, g, 1);
    }
    uint32_t seen_load = 0;
    const uint32_t l32 = lane & 31u, lhi = lane >> 5;
    // Swizzled byte offset of this lane's 16-byte chunk in k-half 0 of its
    // first A row; k-half 1 is the same offset XOR 32 (chunk lhi ^ 2).  Row
    // blocks 32 rows apart lie 2048 bytes apart with the same swizzle, and
    // the lane's B row (wn * 64 + l32) has the A row's swizzle too, so its
    // offset is the A offset plus a wave-uniform distance: one per-lane
    // register serves every fragment address.
    const uint32_t arow = wm * 128u + l32;
    const uint32_t a_off0 = swz(arow, lhi);
    const uint32_t b_dist = kSlotBytes / 2 + (wn * 64u - wm * 128u) * 64u;   // B slot half + row distance
    uint32_t slot = 0;
    // Fragments of one k-half (4 A row blocks, 2 B column blocks) live in
    // registers.  mma_half issues the 8 MFMAs of the fragments held and, when
    // it refills, replaces each A fragment with k-half h of ring slot sl as
    // soon as its two MFMAs are issued and the B pair after the last row
    // block, so the next k-half's LDS reads run under these MFMAs; the
    // scheduling barriers keep the compiler from hoisting the refills (a
    // second register set) or sinking them.
    auto rd_at = [](uint32_t addr, uint32_t imm) {
      return __builtin_bit_cast(bf16x8, *(const BFS_LDS u32x4 *)(uintptr_t)(addr + imm));
    };
    bf16x8 fa[4], fb0, fb1;
    auto read_half = [&](uint32_t sl, int h) __attribute__((always_inline)) {
      const uint32_t a_addr = (a_off0 ^ (32u * h)) + ring_base + sl * kSlotBytes;
      fb0 = rd_at(a_addr + b_dist, 0u);
      fb1 = rd_at(a_addr + b_dist, 2048u);
#pragma unroll
      for (int bm = 0; bm < 4; ++bm) fa[bm] = rd_at(a_addr, 2048u * bm);
    };
    auto mma_half = [&](auto refill, uint32_t sl, int h) __attribute__((always_inline)) {
#pragma unroll
      for (int bm = 0; bm < 4; ++bm) {
        acc[bm * 2 + 0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb0, fa[bm], acc[bm * 2 + 0], 0, 0, 0);
        acc[bm * 2 + 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb1, fa[bm], acc[bm * 2 + 1], 0, 0, 0);
        if constexpr (decltype(refill)::value) {
          const uint32_t a_addr = (a_off0 ^ (32u * h)) + ring_base + sl * kSlotBytes;
          fa[bm] = rd_at(a_addr, 2048u * bm);
          if (bm == 3) {
            fb0 = rd_at(a_addr + b_dist, 0u);
            fb1 = rd_at(a_addr + b_dist, 2048u);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    using Refill = std::true_type;
    using NoRefill = std::false_type;
    auto mma_step = [&](uint32_t it) __attribute__((always_inline)) {
      if (kFlat) {
        S.wait_fixed((uint32_t)P.c_load, kLoadW, it + 2u, P.dep_mma[it], 0u, seen_load, [] {});
      } else {
        g.r1 += 1;
        g.h1 = it + 1;
        S.wait_affine(s_mma, P.mma, g, it + 1, g.r1 - 1, [] {});
      }
      if (!S.aborted) {
        read_half(slot, 0);
        mma_half(Refill{}, slot, 1);
        // every fragment read of the step is issued: MMA retires from the
        // slot (LDS executes this wave's reads before the signal that
        // follows them; the remaining MFMAs use registers only)
        S.signal(P.mma.update, ew);
        mma_half(NoRefill{}, slot, 0);
      } else {
        S.signal(P.mma.update, ew);
      }
      if (!kFlat) S.sync_point(S.word(1, ew));              // end of a K iteration (barrier mode)
      slot = (slot + 1 == (uint32_t)P.ring) ? 0u : slot + 1;
    };
    if constexpr (kFlat) {
#pragma unroll
      for (int st = 0; st < kSteps; ++st) mma_step((uint32_t)st);
    } else {
      uint32_t it = 0;
      for (; it + kUnroll <= trip_k; it += kUnroll) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) mma_step(it + u);
      }
      for (; it < trip_k; ++it) mma_step(it);
    }
    k_end = S.elapsed();
    S.sync_point(S.word(1, ew));                            // before loop C
    S.enter(s_spill, P.spill, g, LC);
    // The chunk loop is unrolled so that each chunk names its accumulator
    // block statically; trip_c <= 8 chunks run.
#pragma unroll
    for (uint32_t it = 0; it < 8; ++it) {
      if (it >= trip_c) break;
      c_iter(it);
      S.wait(s_spill, P.spill, g, it + 1, c_r() - 1, [] {});
      if (!S.aborted) {
        const uint32_t b = it, bm = b >> 1, bn = b & 1u;
        const uint32_t eslot = it & (uint32_t)(P.e_ring - 1);   // e_ring is a power of two
        const uint32_t blk = ering_base + eslot * kESlotBytes + ew * 2048u;
        const f32x16 v = acc[it];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t ncol = wn * 64u + bn * 32u + 8u * j + 4u * lhi;   // first of 4 columns
          const f32x4 bb = *(const BFS_LDS f32x4 *)(uintptr_t)(lds_addr(bias_l) + 4u * ncol);
          const float x0 = gelu_erf(v[4 * j + 0] + bb.x), x1 = gelu_erf(v[4 * j + 1] + bb.y);
          const float x2 = gelu_erf(v[4 * j + 2] + bb.z), x3 = gelu_erf(v[4 * j + 3] + bb.w);
          const bf16x2 p01 = __builtin_convertvector(f32x2{x0, x1}, bf16x2);
          const bf16x2 p23 = __builtin_convertvector(f32x2{x2, x3}, bf16x2);
          const u32x2 q = {__builtin_bit_cast(uint32_t, p01), __builtin_bit_cast(uint32_t, p23)};
          *(BFS_LDS u32x2 *)(uintptr_t)(blk + l32 * 64u + (8u * j + 4u * lhi) * 2u) = q;
        }
        (void)bm;
      }
      S.signal(P.spill.update, ew);
      S.sync_point(S.word(1, ew));                          // end of a C iteration
    }
  } else {
    // -------------------------------------------------------- epilogue engine
    const uint32_t ew = (uint32_t)(wave - kLoadW - kMmaW);
    Site<1> s_epi;
    if (!kFlat) {
      S.sync_point(S.word(2, ew));                          // before loop K
      for (uint32_t it = 0; it < trip_k; ++it) {
        g.r1 += 1;
        g.h1 = it + 1;
        S.sync_point(S.word(2, ew));                        // end of a K iteration
      }
    }
    S.sync_point(S.word(2, ew));                            // before loop C
    S.enter(s_epi, P.epi, g, LC);
    for (uint32_t it = 0; it < trip_c; ++it) {
      c_iter(it);
      S.wait_affine(s_epi, P.epi, g, it + 1, c_r() - 1, [] {});
      if (!S.aborted) {
        const uint32_t b = it, bm = b >> 1, bn = b & 1u;
        const uint32_t eslot = it & (uint32_t)(P.e_ring - 1);   // e_ring is a power of two
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t v = ew * 4u + q;              // MFMA wave whose block this is
          const uint32_t vm = v >> 2, vn = v & 3u;
          const uint32_t blk = ering_base + eslot * kESlotBytes + v * 2048u;
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const uint32_t row = 16u * h + (lane >> 2), cc = lane & 3u;
            const u32x4 d = *(const BFS_LDS u32x4 *)(uintptr_t)(blk + row * 64u + cc * 16u);
            const size_t gm = (size_t)m0 + vm * 128u + bm * 32u + row;
            const size_t gn = (size_t)n0 + vn * 64u + bn * 32u + 8u * cc;
            *reinterpret_cast<u32x4 *>(P.c + gm * P.n + gn) = d;
          }
        }
      }
      S.signal(P.epi.update, ew);
      S.sync_point(S.word(2, ew));                          // end of a C iteration
    }
  }
  drain_all();
  S.finish(lane, k_end);
}

}  // namespace

namespace bfs {

bfs_status launch_gemm(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                       const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream, uint32_t *dbg,
                       int64_t dbg_cap, const bfs_run_opts &o) {
  // structure: top{ BIAS(E0); K{ LOAD(E0) MMA(E1) }; C{ SPILL(E1) EPI(E2) } }, or the K-unrolled
  // top{ BIAS(E0); LOAD_0(E0) MMA_0(E1) ... LOAD_{S-1} MMA_{S-1}; C{ SPILL(E1) EPI(E2) } }
  const bool flat = p->n_loops == 2;
  const int LC = flat ? 1 : 2;
  if (flat ? p->loop_parent[1] != 0 : (p->n_loops != 3 || p->loop_parent[1] != 0 || p->loop_parent[2] != 0))
    return fail(BFS_E_UNSUPPORTED, "gemm: loops must be top -> K, top -> C (or top -> C with K unrolled)");
  if (p->n_engines != 3 || p->waves_per_engine[0] != kLoadW || p->waves_per_engine[1] != kMmaW ||
      p->waves_per_engine[2] != kEpiW)
    return fail(BFS_E_UNSUPPORTED, "gemm: engines of 2, 8 and 2 waves");
  int ins_bias = -1, ins_load = -1, ins_mma = -1, ins_spill = -1, ins_epi = -1;
  std::vector<int> loads, mmas;   // K-unrolled: step s's instructions in listing order
  for (size_t i = 0; i < p->instr_engine.size(); ++i) {
    const int op = p->instr_opcode[i], e = p->instr_engine[i], par = p->instr_parent[i];
    if (op == 20 && e == 0 && par == 0 && ins_bias < 0) ins_bias = (int)i;
    else if (op == 16 && e == 0 && par == (flat ? 0 : 1) && (flat || ins_load < 0)) loads.push_back((int)i), ins_load = (int)i;
    else if (op == 17 && e == 1 && par == (flat ? 0 : 1) && (flat || ins_mma < 0)) mmas.push_back((int)i), ins_mma = (int)i;
    else if (op == 18 && e == 1 && par == LC && ins_spill < 0) ins_spill = (int)i;
    else if (op == 19 && e == 2 && par == LC && ins_epi < 0) ins_epi = (int)i;
    else return fail(BFS_E_UNSUPPORTED, "gemm: unexpected instruction " + std::to_string(i));
  }
  if (ins_bias < 0 || ins_load < 0 || ins_mma < 0 || ins_spill < 0 || ins_epi < 0)
    return fail(BFS_E_UNSUPPORTED, "gemm: needs BIAS, LOAD, MMA, SPILL and EPI");
  const int32_t *la = &p->instr_args[8 * loads[0]];
  const int M = la[0], N = la[1], K = la[2], ring = la[3];
  const int e_ring = p->instr_args[8 * ins_spill];
  if (M <= 0 || N <= 0 || K <= 0 || M % kTile || N % kTile || K % kBK)
    return fail(BFS_E_UNSUPPORTED, "gemm: M and N must be multiples of 256, K a multiple of 32");
  if ((uint64_t)kTile * K * 2 > 0xffffffffull) return fail(BFS_E_UNSUPPORTED, "gemm: K too large for 32-bit load offsets");
  if (ring < 2 || ring > 4 || e_ring < 1 || e_ring > 8 || (e_ring & (e_ring - 1)))
    return fail(BFS_E_UNSUPPORTED, "gemm: ring of 2..4 slots, epilogue ring of 1, 2, 4 or 8 slots");
  if ((M / kTile) * (N / kTile) != n_wg) return fail(BFS_E_INVALID, "gemm: n_wg must be (M / 256) * (N / 256)");
  if (nbufs < 4 || !bufs[0] || !bufs[1] || !bufs[2] || !bufs[3]) return fail(BFS_E_INVALID, "gemm: needs [A, Bt, bias, C]");
  if (!trips || !trip_off) return fail(BFS_E_INVALID, "gemm: needs trip tables");
  const std::vector<DevWait> dw = device_waits(p);
  GemmParams P{};
  P.n_loops = p->n_loops;
  const int steps = K / kBK;
  if (flat) {
    // the K-unrolled program: its K-phase waits are the static immediates
    // the kernel is built with; check the plan gives exactly those
    if ((int)loads.size() != steps || (int)mmas.size() != steps || (steps != 3 && steps != 8 && steps != 128))
      return fail(BFS_E_UNSUPPORTED, "gemm: the K-unrolled kernel is built for 3, 8 or 128 steps, one LOAD and MMA each");
    for (int st = 0; st < steps; ++st) {
      const int32_t *a = &p->instr_args[8 * loads[st]];
      if (a[0] != M || a[1] != N || a[2] != K || a[3] != ring || a[4] != st || p->instr_args[8 * mmas[st]] != st)
        return fail(BFS_E_UNSUPPORTED, "gemm: K-unrolled steps out of order");
    }
    if (p->instr_update[ins_bias] != p->instr_update[loads[0]])
      return fail(BFS_E_UNSUPPORTED, "gemm: BIAS and the LOADs must share the load engine's top-level counter");
    P.c_load = p->instr_update[loads[0]];
    P.c_mma = p->instr_update[mmas[0]];
    for (int st = 0; st < steps; ++st) {
      if (p->instr_update[loads[st]] != P.c_load || p->instr_update[mmas[st]] != P.c_mma)
        return fail(BFS_E_UNSUPPORTED, "gemm: every step must update the engine's top-level counter");
      auto check = [&](int ins, int want_prd, int want_slot, uint32_t want_thr, uint16_t &dep_out) -> bool {
        int n = 0;
        for (int wi = p->instr_wait_off[ins]; wi < p->instr_wait_off[ins + 1]; ++wi) {
          const int d = p->instr_wait_list[wi];
          uint32_t thr = 0;
          if (bfs_eval_threshold(p, d, 1u, 1u, &thr) != BFS_OK) return false;
          if (p->deps[3 * d] != want_prd || dw[d].counter != want_slot || thr != want_thr || !dw[d].active) return false;
          dep_out = (uint16_t)d;
          ++n;
        }
        return want_prd < 0 ? n == 0 : n == 1;
      };
      if (!check(mmas[st], loads[st], P.c_load, (uint32_t)st + 2u, P.dep_mma[st]))
        return fail(BFS_E_UNSUPPORTED, "gemm: MMA " + std::to_string(st) + " must wait exactly for LOAD " +
                                           std::to_string(st) + " (load counter " + std::to_string(st + 2) + ")");
      const int prd = st >= ring ? mmas[st - ring] : -1;
      if (!check(loads[st], prd, P.c_mma, st >= ring ? (uint32_t)(st - ring + 1) : 0u, P.dep_load[st]))
        return fail(BFS_E_UNSUPPORTED, "gemm: LOAD " + std::to_string(st) + " must wait exactly for MMA " +
                                           std::to_string(st - ring) + " (the ring)");
    }
    if (!has_dep(p, mmas[steps - 1], ins_spill, 0) || (size_t)e_ring * kESlotBytes > (size_t)ring * kSlotBytes)
      return fail(BFS_E_UNSUPPORTED, "gemm: needs the last MMA -> SPILL dependency (epilogue ring reuses the K ring)");
    ins_load = loads[0];
    ins_mma = mmas[0];
  } else {
    // the epilogue ring lives in the K ring's memory: the program must order
    // every spill after the whole K loop of every MFMA wave
    if (!has_dep(p, ins_mma, ins_spill, 0) || (size_t)e_ring * kESlotBytes > (size_t)ring * kSlotBytes)
      return fail(BFS_E_UNSUPPORTED, "gemm: needs the MMA -> SPILL dependency (epilogue ring reuses the K ring)");
    if (!fill_waits(p, dw, ins_load, P.load) || !fill_waits(p, dw, ins_mma, P.mma))
      return fail(BFS_E_RESOURCE, "gemm: at most 4 waits per instruction");
  }
  if (!fill_waits(p, dw, ins_bias, P.bias) || !fill_waits(p, dw, ins_spill, P.spill) || !fill_waits(p, dw, ins_epi, P.epi))
    return fail(BFS_E_RESOURCE, "gemm: at most 4 waits per instruction");
  P.load.update = p->instr_update[ins_load];
  P.mma.update = p->instr_update[ins_mma];
  if (!waits_fit({{&P.bias, 1}, {&P.load, 1}, {&P.mma, 1}, {&P.spill, 3}, {&P.epi, 1}}))
    return fail(BFS_E_RESOURCE, "gemm: more waits on an instruction than its engine loop takes");
  if (p->mode == BFS_MODE_BARRIER_FREE && ((!flat && (!no_dynamic(P.load) || !no_dynamic(P.mma))) || !no_dynamic(P.epi)))
    return fail(BFS_E_UNSUPPORTED, "gemm: a K- or C-loop wait depends on a loop register other than its own loop's");
  P.a = static_cast<const __bf16 *>(bufs[0]);
  P.bt = static_cast<const __bf16 *>(bufs[1]);
  P.bias_v = static_cast<const float *>(bufs[2]);
  P.c = static_cast<__bf16 *>(const_cast<void *>(bufs[3]));
  P.trips = trips;
  P.trip_off = trip_off;
  P.sc = sync_common(img, dbg, dbg_cap, o, kWaves);
  P.m = M;
  P.n = N;
  P.k = K;
  P.ring = ring;
  P.e_ring = e_ring;
  P.tiles_m = M / kTile;
  P.tiles_n = N / kTile;
  P.xcd_map = (n_wg % 8 == 0 && P.tiles_m % 4 == 0 && P.tiles_n % 2 == 0) ? 1 : 0;
  const size_t lds = kCntBytes + (size_t)ring * kSlotBytes + 1024;
  const bool instr = dbg || o.dev_stats || o.fault_dep >= 0;
  hipStream_t s = (hipStream_t)stream;
  auto go = [&](auto kern) -> bfs_status {
    hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("gemm attribute: ") + hipGetErrorString(e));
    hipLaunchKernelGGL(kern, dim3(n_wg), dim3(64 * kWaves), lds, s, P);
    e = hipGetLastError();
    if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("gemm launch: ") + hipGetErrorString(e));
    return BFS_OK;
  };
  // Instrumented launches (debug log, statistics, injected faults) run the
  // same unrolled bodies as timed ones, so the debug log records the waits
  // of the code path that is timed.
  auto pick = [&](auto mode_tag, auto instr_tag) -> bfs_status {
    constexpr int kM = decltype(mode_tag)::value;
    constexpr bool kI = decltype(instr_tag)::value;
    if (flat) {
      if (steps == 3) return go(gemm_kernel<kM, kI, 1, 3>);
      if (steps == 8) return go(gemm_kernel<kM, kI, 1, 8>);
      return go(gemm_kernel<kM, kI, 1, 128>);
    }
    switch (o.k_unroll) {
      case 2: return go(gemm_kernel<kM, kI, 2, 0>);
      case 4: return go(gemm_kernel<kM, kI, 4, 0>);
      case 8: return go(gemm_kernel<kM, kI, 8, 0>);
      default: return go(gemm_kernel<kM, kI, 1, 0>);
    }
  };
  using BF = std::integral_constant<int, BFS_MODE_BARRIER_FREE>;
  using BB = std::integral_constant<int, BFS_MODE_BARRIER>;
  if (p->mode == BFS_MODE_BARRIER) return instr ? pick(BB{}, std::true_type{}) : pick(BB{}, std::false_type{});
  return instr ? pick(BF{}, std::true_type{}) : pick(BF{}, std::false_type{});
}

}  // namespace bfs
