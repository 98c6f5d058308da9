// MoE grouped GEMM with top-1 routing, two launches per layer, three engines
// per workgroup, one workgroup per (expert, N-tile, run of M-tiles of BM token
// rows, BM = 128 or 256):
//
//   phase 1  h[rows of expert e][n0 .. n0 + 127] = SiLU(x W_gate) * (x W_up),
//            token rows gathered from x through the expert-grouped
//            permutation, h stored bf16 in grouped row order;
//   phase 2  y[token][n0 .. n0 + 255] = h W_down, rows scattered back to
//            their tokens.
//
//   E0 (2 waves, load)      ACQL at each M-tile; LOAD: the step's BM token
//                           rows (wave 0) and 256 weight rows (wave 1), 32
//                           wide in K, into a ring slot with direct-to-LDS
//                           loads.
//   E1 (8 waves, MFMA)      MMA: a BM / 2-row sub-tile per wave, fp32
//                           accumulators (phase 1: gate and up for 32 h
//                           columns, so SiLU(g) * u needs no exchange;
//                           phase 2: 64 y columns); ACQE at each M-tile;
//                           SPILL: one 32 x 32 block per chunk, packed to
//                           bf16 into an epilogue slot.
//   E2 (2 waves, epilogue)  EPI: the chunk's 16-byte row segments into
//                           registers, then to HBM (at 256-row tiles with at
//                           most one epilogue slot, retiring before the
//                           stores).
//
// The M loop runs the workgroup's M-tiles, a count derived from the routing
// and known only at run time; K runs K / 32 steps, C BM / 64 (phase 1) or
// BM / 32 (phase 2) chunks per M-tile.  Dependencies: LOAD->MMA (k = 0),
// MMA->LOAD (k = ring), SPILL->EPI (k = 0), EPI->ACQE (k = 1, C3), and one of
// two epilogue layouts:
//   * epilogue slots after the ring: EPI->SPILL (k = epilogue slots) and
//     MMA->ACQL (k = 1, C3: an M-tile's loads start after the previous
//     tile's MFMAs released the ring);
//   * epilogue in the ring (epilogue ring 0): every chunk of an M-tile has
//     its own 16 KiB of the ring, MMA->SPILL (k = 0, C2: the spills start
//     after the tile's last MFMAs read the ring) and EPI->ACQL (k = 1, C3:
//     the next tile's loads start after the epilogue read its chunks), so
//     the MFMA engine spills a whole M-tile without waiting for the stores.
// In place of MMA->ACQL the program may read MMA->LOAD with the linearized
// offset (an extension of the paper's relation: k counts K steps over all
// M-tiles of the workgroup), which orders exactly the reuse of ring slot
// (r_K - 1) % ring across M-tiles, so the next tile's loads overlap the
// previous tile's MFMAs.  Token rows past the expert's count are loaded from
// a clamped row and never stored.
//
// LDS (bytes): counters 2048 | ring slots of BM x 64 + 16 KiB (token rows
// BM x 64 B, then weight rows 256 x 64 B; 16-byte chunk c of row r at
// c ^ ((r / 4) % 4))
// | epilogue slots of 16 KiB (8 blocks of 32 x 32 bf16, row-major), unless
// the epilogue lives in the ring.
//
// Family contract (BFS_KERNEL_MOE): loops top -> M -> {K, C}; ACQL (E0, NOP)
// at M before K; LOAD (E0, opcode 48, args [phase, K, N, ring, BM (0: 128)]) and MMA (E1,
// 49) in K; ACQE (E1, NOP) at M between K and C; SPILL (E1, 51, args
// [epilogue slots, 0: in the ring]) and EPI (E2, 50) in C; waves 2, 8, 2.  Phase 1: K = hidden
// (multiple of 32), N = ffn (multiple of 128); phase 2: K = ffn (multiple of
// 32), N = hidden (multiple of 256).  Buffers: [0] work list int32 [n_wg][4]
// = (expert, first output column, first M-tile, M-tiles), [1] perm int32
// [tokens] (token ids grouped by expert), [2] expert_off int32 [experts + 1];
// phase 1: [3] x bf16 [tokens][hidden], [4] W_gate, [5] W_up bf16
// [experts][ffn][hidden], [6] h bf16 [tokens][ffn]; phase 2: [3] h, [4]
// W_down bf16 [experts][hidden][ffn], [5] y bf16 [tokens][hidden].
#include <string>
#include <type_traits>

#include "engine_sync.h"

using namespace bfsdev;

namespace {

constexpr int kBK = 32;
constexpr int kLoadW = 2, kMmaW = 8, kEpiW = 2, kWaves = 12;
// ring slot: the token rows of one K step (8 KiB for M-tiles of 128 rows,
// 16 KiB for 256), then 256 weight rows (16 KiB)
constexpr uint32_t a_slot_bytes(int bm) { return (uint32_t)bm * kBK * 2; }
constexpr uint32_t slot_bytes(int bm) { return a_slot_bytes(bm) + 256 * kBK * 2; }
constexpr uint32_t kESlotBytes = kMmaW * 32 * 32 * 2;

struct MoeParams {
  SyncCommon sc;
  InstrWaits acql, load, mma, acqe, spill, epi;
  const int32_t *work;
  const int32_t *perm;
  const int32_t *eoff;
  const __bf16 *a;          // x (phase 1) or h (phase 2)
  const __bf16 *w0;         // W_gate (phase 1) or W_down (phase 2)
  const __bf16 *w1;         // W_up (phase 1)
  __bf16 *out;              // h (phase 1) or y (phase 2)
  const int32_t *trips;
  const int64_t *trip_off;
  int32_t kdim, ndim, ring, e_ring, n_experts, n_tokens;
};

__device__ __forceinline__ uint32_t swz(uint32_t row, uint32_t chunk) {
  return row * 64u + ((chunk ^ ((row >> 2) & 3u)) << 4);
}

__device__ __forceinline__ float silu(float g) { return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)); }

// kBM: token rows per M-tile.  128: each MFMA wave holds a 64-row sub-tile
// (two row blocks); 256: a 128-row sub-tile (four row blocks), twice the MFMA
// work per K step and per synchronization, half the weight re-reads.
template <int kPhase, int kMode, bool kInstr, int kBM>
__global__ void __launch_bounds__(768) moe_kernel(MoeParams P) {
  constexpr uint32_t kASlot = a_slot_bytes(kBM), kSlotBytes = slot_bytes(kBM);
  constexpr int kRB = kBM / 64;                     // 32-row blocks per MFMA wave
  constexpr uint32_t kChunks = kPhase == 1 ? (uint32_t)kRB : 2u * kRB;
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  uint32_t *cnt = reinterpret_cast<uint32_t *>(lds);
  const uint32_t ring = lds_addr(lds) + kCntBytes;
  // epilogue slots: after the ring, or (e_ring 0) the ring's own memory,
  // one 16 KiB slot per chunk, free once the M-tile's K loop is over
  const uint32_t ering = P.e_ring == 0 ? ring : ring + (uint32_t)P.ring * kSlotBytes;
  for (int i = threadIdx.x; i < bfs::kMaxSlots * bfs::kMaxWavesPerEngine; i += blockDim.x) cnt[i] = 0;
  __syncthreads();

  const int wave = wave_id();
  const uint32_t lane = lane_id(), l32 = lane & 31u, lhi = lane >> 5;
  const int wg = blockIdx.x;
  Sync<kMode, kInstr> S(P.sc, lds_addr(cnt), wave, wg);

  const int32_t expert = ldc(P.work + 4 * wg + 0), n0 = ldc(P.work + 4 * wg + 1);
  const int32_t mt0 = ldc(P.work + 4 * wg + 2);
  const int32_t e_lo = ldc(P.eoff + expert), e_cnt = ldc(P.eoff + expert + 1) - e_lo;
  const int64_t *toff = P.trip_off + (int64_t)wg * 4;
  uint32_t trip_m = (uint32_t)ldc(P.trips + ldc(toff + 1));
  const int64_t k_off = ldc(toff + 2), c_off = ldc(toff + 3);
  const uint32_t ksteps = (uint32_t)(P.kdim / kBK), chunks = kChunks;
  const uint32_t max_m = (uint32_t)max(0, (e_cnt + kBM - 1) / kBM - mt0);
  if (trip_m > max_m) {
    report_input(P.sc.err, 1u, (uint32_t)wg, 1u, trip_m, max_m, (uint32_t)wave);
    trip_m = max_m;
  }
  Regs g;
  Site<1> sa, sb, sc;               // one per wait site of the engine (each has one wait)
  uint64_t mark = 0;

  if (wave < kLoadW) {
    // ------------------------------------------------------------ load engine
    const uint32_t ew = (uint32_t)wave;
    constexpr int kALoads = kBM / 16;                          // token-row loads per step (16 rows each)
    const int per_group = wave == 0 ? kALoads : 16;           // loads per step
    int pending = 0;
    auto retire_one = [&]() {
      if (pending == 3) {
        if (per_group == 8) wait_vm<16>(); else wait_vm<32>();
      } else if (pending == 2) {
        if (per_group == 8) wait_vm<8>(); else wait_vm<16>();
      } else {
        wait_vm<0>();
      }
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
    // lane l covers rows 16 j + l / 4 and the 16-byte chunk that belongs at
    // position l % 4 of its row
    const uint32_t r_in = lane >> 2, chunk = (lane & 3u) ^ ((lane >> 4) & 3u);
    // phase 1: the token ids of an M-tile's rows (gathered through perm)
    // are loaded during the previous M-tile, so a tile's first row loads
    // need not wait for them.  These loads are older than the ring loads
    // issued after them, so the counted vmcnt waits below only wait longer
    // for them, never shorter.
    int32_t prow[kALoads];
    auto load_rows = [&](uint32_t mi) __attribute__((always_inline)) {
      const int32_t m0 = (mt0 + (int32_t)mi) * kBM;
#pragma unroll
      for (int j = 0; j < kALoads; ++j) {
        const int32_t r = min(m0 + 16 * j + (int32_t)r_in, e_cnt - 1);
        prow[j] = kPhase == 1 ? P.perm[e_lo + r] : e_lo + r;
      }
    };
    if (wave == 0 && trip_m > 0) load_rows(0);
    S.sync_point(S.word(0, ew));                                  // before loop M
    S.enter(sa, P.acql, g, 1);
    for (uint32_t mi = 0; mi < trip_m; ++mi) {
      g.r1 += 1;
      g.h1 = mi + 1;
      S.wait(sa, P.acql, g, mi + 1, g.r1 - 1, [&] { if (pending > 0) retire_one(); });   // ACQL
      S.signal(P.acql.update, ew);
      retire_all();
      // the K and C loops have static trips; a trip table that disagrees is
      // reported (the static trips run)
      if (wave == 0) {
        const int32_t tk = ldc(P.trips + k_off + mi), tc = ldc(P.trips + c_off + mi);
        if (tk != (int32_t)ksteps || tc != (int32_t)chunks)
          report_input(P.sc.err, 2u, (uint32_t)wg, mi, (uint32_t)tk, (uint32_t)tc, (uint32_t)wave);
      }
      const int32_t m0 = (mt0 + (int32_t)mi) * kBM;
      // source rows of this M-tile as 32-bit per-lane byte offsets from a
      // wave-uniform base that advances one K step per iteration: the loads
      // take the scalar-base address form and need no vector address
      // arithmetic (which would compete for issue with the MFMA waves)
      uint32_t voff[16];
      if (wave == 0) {
#pragma unroll
        for (int j = 0; j < kALoads; ++j) {
          const int32_t row = prow[j];
          const uint64_t off = ((uint64_t)(uint32_t)row * (uint32_t)P.kdim + 8u * chunk) * 2u;
          if (__ballot((off >> 32) != 0) != 0ull) {
            report_input(P.sc.err, 3u, (uint32_t)wg, mi, (uint32_t)row, 0u, (uint32_t)wave);
            S.aborted = 1u;
          }
          voff[j] = (uint32_t)off;
        }
#pragma unroll
        for (int j = kALoads; j < 16; ++j) voff[j] = 0u;
        if (mi + 1 < trip_m) load_rows(mi + 1);
      } else {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const uint32_t r = 16u * j + r_in;
          const uint32_t n = kPhase == 1 ? (n0 + (r & 127u)) : (n0 + r);
          voff[j] = (n * (uint32_t)P.kdim + 8u * chunk) * 2u;      // within the expert's matrix
        }
      }
      S.sync_point(S.word(0, ew));                                // before loop K
      S.enter(sb, P.load, g, 2);
      uint32_t slot = (g.r2) % (uint32_t)P.ring;
      for (uint32_t it = 0; it < ksteps; ++it, slot = (slot + 1 == (uint32_t)P.ring) ? 0u : slot + 1) {
        g.r2 += 1;
        g.h2 = it + 1;
        S.wait_affine(sb, P.load, g, it + 1, g.r2 - 1, [&] { if (pending > 0) retire_one(); });
        if (!S.aborted) {
          const uint32_t dst = ring + slot * kSlotBytes + (wave == 0 ? 0u : kASlot);
          const size_t kb = (size_t)it * (kBK * 2);
          if (wave == 0) {
            const char *sb = reinterpret_cast<const char *>(P.a) + kb;
#pragma unroll
            for (int j = 0; j < kALoads; ++j) {
              asm volatile("" : "+v"(voff[j]));   // keep the offset a 32-bit value at its use
              __builtin_amdgcn_global_load_lds((const void *)(sb + voff[j]), (BFS_LDS void *)(uintptr_t)(dst + 1024u * j),
                                               16, 0, 0);
            }
          } else {
            // phase 1: weight rows 0..127 are W_gate's, 128..255 W_up's
            const size_t eb = (size_t)expert * P.ndim * P.kdim * 2 + kb;
            const char *sb0 = reinterpret_cast<const char *>(P.w0) + eb;
            const char *sb1 = kPhase == 1 ? reinterpret_cast<const char *>(P.w1) + eb : sb0;
#pragma unroll
            for (int j = 0; j < 16; ++j) {
              asm volatile("" : "+v"(voff[j]));
              __builtin_amdgcn_global_load_lds((const void *)((j < 8 ? sb0 : sb1) + voff[j]),
                                               (BFS_LDS void *)(uintptr_t)(dst + 1024u * j), 16, 0, 0);
            }
          }
          pending += 1;
          if (pending == 3) retire_one();
        } else {
          S.signal(P.load.update, ew);
        }
        if (kMode == BFS_MODE_BARRIER) {
          retire_all();
          S.sync_point(S.word(0, ew));                            // end of a K iteration
        }
      }
      retire_all();
      S.sync_point(S.word(0, ew));                                // before loop C
      for (uint32_t c = 0; c < chunks; ++c) {
        g.r3 += 1;
        g.h3 = c + 1;
        S.sync_point(S.word(0, ew));                              // end of a C iteration
      }
      S.sync_point(S.word(0, ew));                                // end of an M iteration
    }
  } else if (wave < kLoadW + kMmaW) {
    // ------------------------------------------------------------ MFMA engine
    const uint32_t ew = (uint32_t)(wave - kLoadW);
    const uint32_t wm = ew >> 2, wn = ew & 3u;
    const uint32_t arow = wm * (uint32_t)(kBM / 2) + l32;
    // weight rows of the two column blocks of this wave
    const uint32_t brow0 = kPhase == 1 ? 32u * wn + l32 : 64u * wn + l32;
    const uint32_t brow1 = kPhase == 1 ? 128u + 32u * wn + l32 : 64u * wn + 32u + l32;
    // swizzled byte offsets of this lane's 16-byte chunk in k-half 0 and 1;
    // row blocks 32 rows apart are 2048 bytes apart with the same swizzle,
    // and brow1 lies b_step bytes after brow0 (a multiple of 16 rows)
    const uint32_t a_off[2] = {swz(arow, lhi), swz(arow, 2u + lhi)};
    const uint32_t b_off[2] = {swz(brow0, lhi), swz(brow0, 2u + lhi)};
    constexpr uint32_t b_step = kPhase == 1 ? 128u * 64u : 32u * 64u;
    auto rd_at = [](uint32_t addr, uint32_t imm) {
      return __builtin_bit_cast(bf16x8, *(const BFS_LDS u32x4 *)(uintptr_t)(addr + imm));
    };
    S.sync_point(S.word(1, ew));                                  // before loop M
    S.enter(sb, P.acqe, g, 1);
    for (uint32_t mi = 0; mi < trip_m; ++mi) {
      g.r1 += 1;
      g.h1 = mi + 1;
      f32x16 acc[2 * kRB];           // [b * kRB + rb]: b = weight block (gate / up, or column block), rb = row block
#pragma unroll
      for (int i = 0; i < 2 * kRB; ++i) acc[i] = f32x16{};
      S.sync_point(S.word(1, ew));                                // before loop K
      S.enter(sa, P.mma, g, 2);
      uint32_t slot = g.r2 % (uint32_t)P.ring;
      for (uint32_t it = 0; it < ksteps; ++it, slot = (slot + 1 == (uint32_t)P.ring) ? 0u : slot + 1) {
        g.r2 += 1;
        g.h2 = it + 1;
        S.wait_affine(sa, P.mma, g, it + 1, g.r2 - 1, [] {});
        if (!S.aborted) {
          const uint32_t a_base = ring + slot * kSlotBytes, b_base = a_base + kASlot;
          auto rd = [&](uint32_t base, uint32_t row, uint32_t c) {
            return __builtin_bit_cast(bf16x8, *(const BFS_LDS u32x4 *)(uintptr_t)(base + swz(row, c)));
          };
          if constexpr (kBM == 128) {
            bf16x8 a0 = rd(a_base, arow, lhi), a1 = rd(a_base, arow + 32u, lhi);
            bf16x8 b0 = rd(b_base, brow0, lhi), b1 = rd(b_base, brow1, lhi);
            const bf16x8 a0n = rd(a_base, arow, 2u + lhi), a1n = rd(a_base, arow + 32u, 2u + lhi);
            const bf16x8 b0n = rd(b_base, brow0, 2u + lhi), b1n = rd(b_base, brow1, 2u + lhi);
            // MMA retires from the slot once its fragments are read: LDS
            // executes this wave's reads before the signal that follows them,
            // and the MFMAs below use registers only
            S.signal(P.mma.update, ew);
            acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b0, a0, acc[0], 0, 0, 0);
            acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b0, a1, acc[1], 0, 0, 0);
            acc[2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b1, a0, acc[2], 0, 0, 0);
            acc[3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b1, a1, acc[3], 0, 0, 0);
            acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b0n, a0n, acc[0], 0, 0, 0);
            acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b0n, a1n, acc[1], 0, 0, 0);
            acc[2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b1n, a0n, acc[2], 0, 0, 0);
            acc[3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b1n, a1n, acc[3], 0, 0, 0);
          } else {
            // four row blocks, fragments of one k-half (4 A, 2 B) in
            // registers: each A fragment is refilled with the next k-half's
            // as soon as its two MFMAs are issued, the B pair after the last
            // row block, so the second k-half's LDS reads run under the
            // first k-half's MFMAs; the scheduling barriers keep the compiler
            // from hoisting the refills (which would need a second set of
            // registers) or sinking them behind waits
            const uint32_t a_lo = a_base + a_off[0], a_hi = a_base + a_off[1];
            const uint32_t b_lo = b_base + b_off[0], b_hi = b_base + b_off[1];
            bf16x8 fa[kRB], fb0, fb1;
            fb0 = rd_at(b_lo, 0u);
            fb1 = rd_at(b_lo, b_step);
#pragma unroll
            for (int rb = 0; rb < kRB; ++rb) fa[rb] = rd_at(a_lo, 2048u * rb);
#pragma unroll
            for (int hk = 0; hk < 2; ++hk) {
#pragma unroll
              for (int rb = 0; rb < kRB; ++rb) {
                acc[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb0, fa[rb], acc[rb], 0, 0, 0);
                acc[kRB + rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb1, fa[rb], acc[kRB + rb], 0, 0, 0);
                if (hk == 0) {
                  fa[rb] = rd_at(a_hi, 2048u * rb);
                  if (rb == kRB - 1) {
                    fb0 = rd_at(b_hi, 0u);
                    fb1 = rd_at(b_hi, b_step);
                  }
                }
                __builtin_amdgcn_sched_barrier(0);
              }
              // every fragment read of the step is issued: MMA retires from
              // the slot (LDS executes the reads before the signal)
              if (hk == 0) S.signal(P.mma.update, ew);
            }
          }
        } else {
          S.signal(P.mma.update, ew);
        }
        S.sync_point(S.word(1, ew));                              // end of a K iteration
      }
      mark = S.elapsed();
      S.wait(sb, P.acqe, g, mi + 1, g.r1 - 1, [] {});                    // ACQE
      S.signal(P.acqe.update, ew);
      S.sync_point(S.word(1, ew));                                // before loop C
      S.enter(sc, P.spill, g, 3);
#pragma unroll
      for (uint32_t c = 0; c < kChunks; ++c) {
        g.r3 += 1;
        g.h3 = c + 1;
        S.wait_affine(sc, P.spill, g, c + 1, g.r3 - 1, [] {});
        if (!S.aborted) {
          const uint32_t eslot = P.e_ring == 0 ? c : (P.e_ring == 2 ? ((g.r3 - 1) & 1u) : 0u);
          const uint32_t blk = ering + eslot * kESlotBytes + ew * 2048u;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              if (kPhase == 1) v[e] = silu(acc[c][4 * j + e]) * acc[kRB + c][4 * j + e];   // chunk = row block
              else v[e] = acc[(c & 1u) * kRB + (c >> 1)][4 * j + e];                      // chunk = rb * 2 + cb
            }
            const u32x2 q = {__builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{v[0], v[1]}, bf16x2)),
                             __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{v[2], v[3]}, bf16x2))};
            *(BFS_LDS u32x2 *)(uintptr_t)(blk + l32 * 64u + (8u * j + 4u * lhi) * 2u) = q;
          }
        }
        S.signal(P.spill.update, ew);
        S.sync_point(S.word(1, ew));                              // end of a C iteration
      }
      S.sync_point(S.word(1, ew));                                // end of an M iteration
    }
  } else {
    // -------------------------------------------------------- epilogue engine
    const uint32_t ew = (uint32_t)(wave - kLoadW - kMmaW);
    S.sync_point(S.word(2, ew));                                  // before loop M
    for (uint32_t mi = 0; mi < trip_m; ++mi) {
      g.r1 += 1;
      g.h1 = mi + 1;
      const int32_t m0 = (mt0 + (int32_t)mi) * kBM;
      // this wave stores the blocks of MFMA waves 4 ew .. 4 ew + 3 (rows
      // kBM / 2 * ew ..), lane rows 16 h + lane / 4 of each 32-row block
      int32_t tok[kRB][2];
#pragma unroll
      for (int rb = 0; rb < kRB; ++rb)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int32_t r = m0 + (kBM / 2) * (int32_t)ew + 32 * rb + 16 * h + (int32_t)(lane >> 2);
          tok[rb][h] = r < e_cnt ? (kPhase == 1 ? e_lo + r : P.perm[e_lo + r]) : -1;
        }
      S.sync_point(S.word(2, ew));                                // before loop K
      for (uint32_t it = 0; it < ksteps; ++it) {
        g.r2 += 1;
        g.h2 = it + 1;
        S.sync_point(S.word(2, ew));                              // end of a K iteration
      }
      S.sync_point(S.word(2, ew));                                // before loop C
      S.enter(sa, P.epi, g, 3);
      for (uint32_t c = 0; c < chunks; ++c) {
        g.r3 += 1;
        g.h3 = c + 1;
        S.wait_affine(sa, P.epi, g, c + 1, g.r3 - 1, [] {});
        if (!S.aborted) {
          const uint32_t eslot = P.e_ring == 0 ? c : (P.e_ring == 2 ? ((g.r3 - 1) & 1u) : 0u);
          const uint32_t rb = kPhase == 1 ? c : (c >> 1), cb = kPhase == 1 ? 0u : (c & 1u);
          auto seg = [&](int q, int h) {            // row segment h of MFMA wave ew * 4 + q's block
            const uint32_t blk = ering + eslot * kESlotBytes + (ew * 4u + q) * 2048u;
            const uint32_t row = 16u * h + (lane >> 2), cc = lane & 3u;
            return *(const BFS_LDS u32x4 *)(uintptr_t)(blk + row * 64u + cc * 16u);
          };
          // the chunk's token of each lane row, tok[rb][h], selected without
          // dynamic indexing (and before the lambdas, which must not take
          // the array's address)
          int32_t trow0 = tok[0][0], trow1 = tok[0][1];
#pragma unroll
          for (int i = 1; i < kRB; ++i) {
            trow0 = rb == (uint32_t)i ? tok[i][0] : trow0;
            trow1 = rb == (uint32_t)i ? tok[i][1] : trow1;
          }
          auto store = [&](int q, int h, const u32x4 &d) {
            const uint32_t cc = lane & 3u;
            const int32_t t = h == 0 ? trow0 : trow1;
            const uint32_t col = kPhase == 1 ? (n0 + 32u * q + 8u * cc) : (n0 + 64u * q + 32u * cb + 8u * cc);
            if (t >= 0) {
              u32x4 *dst = reinterpret_cast<u32x4 *>(P.out + (size_t)t * P.ndim + col);
              *dst = d;
            }
          };
          // With one epilogue slot (256-row M-tiles) the chunk's segments go
          // into registers first and EPI retires from the slot once these
          // reads are issued
          // (LDS executes the wave's reads before the signal that follows
          // them), so the next chunk's spill does not wait behind this
          // chunk's global stores.  With two slots the spill of chunk c + 2
          // already overlaps these stores; there each segment is stored as
          // it arrives and EPI retires after the stores (reading everything
          // first measured slower at 128-row tiles).
          bool early = false;
          if constexpr (kBM == 256) early = P.e_ring <= 1;
          if (early) {
            u32x4 d[4][2];
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
              for (int h = 0; h < 2; ++h) d[q][h] = seg(q, h);
            S.signal(P.epi.update, ew);
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
              for (int h = 0; h < 2; ++h) store(q, h, d[q][h]);
          } else {
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
              for (int h = 0; h < 2; ++h) store(q, h, seg(q, h));
            S.signal(P.epi.update, ew);
          }
        } else {
          S.signal(P.epi.update, ew);
        }
        S.sync_point(S.word(2, ew));                              // end of a C iteration
      }
      S.sync_point(S.word(2, ew));                                // end of an M iteration
    }
  }
  drain_all();
  S.finish(lane, mark);
}

}  // namespace

namespace bfs {

bfs_status launch_moe(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                      const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream, uint32_t *dbg,
                      int64_t dbg_cap, const bfs_run_opts &o) {
  // structure: top{ M{ ACQL(E0); K{ LOAD(E0) MMA(E1) }; ACQE(E1); C{ SPILL(E1) EPI(E2) } } }
  if (p->n_loops != 4 || p->loop_parent[1] != 0 || p->loop_parent[2] != 1 || p->loop_parent[3] != 1)
    return fail(BFS_E_UNSUPPORTED, "moe: loops must be top -> M -> {K, C}");
  if (p->n_engines != 3 || p->waves_per_engine[0] != kLoadW || p->waves_per_engine[1] != kMmaW ||
      p->waves_per_engine[2] != kEpiW)
    return fail(BFS_E_UNSUPPORTED, "moe: engines of 2, 8 and 2 waves");
  int acql = -1, load = -1, mma = -1, acqe = -1, spill = -1, epi = -1;
  for (size_t i = 0; i < p->instr_engine.size(); ++i) {
    const int op = p->instr_opcode[i], e = p->instr_engine[i], par = p->instr_parent[i];
    if (op == 0 && e == 0 && par == 1 && acql < 0 && load < 0) acql = (int)i;
    else if (op == 48 && e == 0 && par == 2 && load < 0) load = (int)i;
    else if (op == 49 && e == 1 && par == 2 && mma < 0) mma = (int)i;
    else if (op == 0 && e == 1 && par == 1 && acqe < 0 && mma >= 0) acqe = (int)i;
    else if (op == 51 && e == 1 && par == 3 && spill < 0) spill = (int)i;
    else if (op == 50 && e == 2 && par == 3 && epi < 0) epi = (int)i;
    else return fail(BFS_E_UNSUPPORTED, "moe: unexpected instruction " + std::to_string(i));
  }
  if (acql < 0 || load < 0 || mma < 0 || acqe < 0 || spill < 0 || epi < 0)
    return fail(BFS_E_UNSUPPORTED, "moe: needs ACQL, LOAD, MMA, ACQE, SPILL and EPI");
  const int32_t *la = &p->instr_args[8 * load];
  const int phase = la[0], K = la[1], N = la[2], ring = la[3], bm = la[4] == 0 ? 128 : la[4];
  const int e_ring = p->instr_args[8 * spill];
  if (bm != 128 && bm != 256) return fail(BFS_E_UNSUPPORTED, "moe: M-tiles of 128 or 256 token rows");
  if (phase != 1 && phase != 2) return fail(BFS_E_UNSUPPORTED, "moe: phase 1 or 2");
  if (K <= 0 || K % kBK || N <= 0 || N % (phase == 1 ? 128 : 256))
    return fail(BFS_E_UNSUPPORTED, "moe: K a multiple of 32, N a multiple of 128 (phase 1) or 256 (phase 2)");
  if (ring < 2 || ring > 5 || e_ring < 0 || e_ring > 2)
    return fail(BFS_E_UNSUPPORTED, "moe: ring 2..5, epilogue 1..2 slots or 0 (in the ring)");
  const int chunks = phase == 1 ? bm / 64 : bm / 32;
  if (e_ring == 0 && (size_t)chunks * kESlotBytes > (size_t)ring * slot_bytes(bm))
    return fail(BFS_E_UNSUPPORTED, "moe: the M-tile's chunks do not fit in the ring");
  const size_t lds = kCntBytes + (size_t)ring * slot_bytes(bm) + (size_t)e_ring * kESlotBytes;
  if (lds > 160 * 1024)
    return fail(BFS_E_RESOURCE, "moe: ring and epilogue slots exceed 160 KiB of LDS");
  if ((uint64_t)N * K * 2 > 0xffffffffull) return fail(BFS_E_UNSUPPORTED, "moe: one expert's matrix must stay below 4 GiB");
  // the ring is protected across M-tiles by MMA->ACQL (k = 1), or by reading
  // MMA->LOAD with the linearized offset (slots are indexed by r_K); with
  // the epilogue in the ring (e_ring 0) the spills wait for the M-tile's
  // last MFMAs (MMA->SPILL, k = 0) and the next M-tile's loads for the
  // epilogue's reads (EPI->ACQL, k = 1), which also orders them after the
  // MFMAs; the epilogue slots are otherwise reused by EPI->SPILL (k =
  // e_ring) within an M-tile
  bool ring_linear = false;
  for (size_t d = 0; d < p->deps.size() / 3; ++d)
    if (p->deps[3 * d] == mma && p->deps[3 * d + 1] == load && p->deps[3 * d + 2] == ring && p->dep_linear[d])
      ring_linear = true;
  const bool epi_ok = e_ring == 0 ? (has_dep(p, mma, spill, 0) && has_dep(p, epi, acql, 1))
                                  : has_dep(p, epi, spill, e_ring);
  const bool across = ring_linear || has_dep(p, mma, acql, 1) || (e_ring == 0 && has_dep(p, epi, acql, 1));
  if (!has_dep(p, load, mma, 0) || !has_dep(p, mma, load, ring) || !across || !epi_ok ||
      !has_dep(p, spill, epi, 0) || !has_dep(p, epi, acqe, 1))
    return fail(BFS_E_UNSUPPORTED, "moe: missing a ring or M-tile dependency");
  const int need = phase == 1 ? 7 : 6;
  if (nbufs < need) return fail(BFS_E_INVALID, "moe: too few buffers");
  for (int i = 0; i < need; ++i)
    if (!bufs[i]) return fail(BFS_E_INVALID, "moe: null buffer");
  if (!trips || !trip_off || n_wg <= 0) return fail(BFS_E_INVALID, "moe: needs trip tables and workgroups");
  const std::vector<DevWait> dw = device_waits(p);
  MoeParams P{};
  if (!fill_waits(p, dw, acql, P.acql) || !fill_waits(p, dw, load, P.load) || !fill_waits(p, dw, mma, P.mma) ||
      !fill_waits(p, dw, acqe, P.acqe) || !fill_waits(p, dw, spill, P.spill) || !fill_waits(p, dw, epi, P.epi))
    return fail(BFS_E_RESOURCE, "moe: at most 4 waits per instruction");
  if (!waits_fit({{&P.acql, 1}, {&P.load, 1}, {&P.mma, 1}, {&P.acqe, 1}, {&P.spill, 1}, {&P.epi, 1}}))
    return fail(BFS_E_RESOURCE, "moe: more waits on an instruction than its engine loop takes");
  if (p->mode == BFS_MODE_BARRIER_FREE &&
      (!no_dynamic(P.load) || !no_dynamic(P.mma) || !no_dynamic(P.spill) || !no_dynamic(P.epi)))
    return fail(BFS_E_UNSUPPORTED, "moe: a K- or C-loop wait depends on a loop register other than its own loop's");
  P.sc = sync_common(img, dbg, dbg_cap, o, kWaves);
  P.work = static_cast<const int32_t *>(bufs[0]);
  P.perm = static_cast<const int32_t *>(bufs[1]);
  P.eoff = static_cast<const int32_t *>(bufs[2]);
  P.a = static_cast<const __bf16 *>(bufs[3]);
  P.w0 = static_cast<const __bf16 *>(bufs[4]);
  P.w1 = phase == 1 ? static_cast<const __bf16 *>(bufs[5]) : nullptr;
  P.out = static_cast<__bf16 *>(const_cast<void *>(bufs[phase == 1 ? 6 : 5]));
  P.trips = trips;
  P.trip_off = trip_off;
  P.kdim = K;
  P.ndim = N;
  P.ring = ring;
  P.e_ring = e_ring;
  const bool instr = dbg || o.dev_stats || o.fault_dep >= 0;
  hipStream_t s = (hipStream_t)stream;
  auto go = [&](auto kern) -> bfs_status {
    hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("moe attribute: ") + hipGetErrorString(e));
    hipLaunchKernelGGL(kern, dim3(n_wg), dim3(64 * kWaves), lds, s, P);
    e = hipGetLastError();
    if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("moe launch: ") + hipGetErrorString(e));
    return BFS_OK;
  };
  const bool bar = p->mode == BFS_MODE_BARRIER;
  auto pick = [&](auto ph, auto bmc) -> bfs_status {
    constexpr int kP = decltype(ph)::value, kB = decltype(bmc)::value;
    if (bar)
      return instr ? go(moe_kernel<kP, BFS_MODE_BARRIER, true, kB>) : go(moe_kernel<kP, BFS_MODE_BARRIER, false, kB>);
    return instr ? go(moe_kernel<kP, BFS_MODE_BARRIER_FREE, true, kB>)
                 : go(moe_kernel<kP, BFS_MODE_BARRIER_FREE, false, kB>);
  };
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using B128 = std::integral_constant<int, 128>;
  using B256 = std::integral_constant<int, 256>;
  if (phase == 1) return bm == 128 ? pick(I1{}, B128{}) : pick(I1{}, B256{});
  return bm == 128 ? pick(I2{}, B128{}) : pick(I2{}, B256{});
}

}  // namespace bfs
