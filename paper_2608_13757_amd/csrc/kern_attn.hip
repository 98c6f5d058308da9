// Variable-length attention forward (no causal mask).  A fixed set of
// workgroups (one per compute unit) each runs a run-time list of (sequence,
// head, 128-query tile) work items, with five engines synchronized by LDS
// counters:
//
//   E0 (1 wave, K load)    LOADK: the 64 x 128 bf16 K block of the step into
//                          a K ring slot with direct-to-LDS loads.
//   E1 (2 waves, MFMA)     QK: S = Q K^T for 64 query rows per wave (the
//                          tile's Q rows held in registers for its KV loop),
//                          written as fp32 into an S/P slot.
//   E2 (4 waves, VALU)     SM: online softmax over 32 rows per wave in the
//                          base-2 domain: running max m, rescale factor
//                          alpha = 2^(m_old - m_new), P = 2^(S c - m_new)
//                          written as bf16 over S in place, running sum l.
//   E3 (4 waves, MFMA)     PREAD: the P fragments and alpha of the wave's 32
//                          query rows into registers; PV: O = alpha O + P V
//                          (fp32 accumulators); after each tile's KV loop
//                          NORM: O / l to HBM.
//   E4 (1 wave, V load)    LOADV: the V block into a V ring slot.
//
// Loops top -> T -> KV: T runs the workgroup's tiles, KV ceil(L / 64) steps
// of a tile; both trips are known only at run time.  Dependencies (the
// program's; Eq. 5 on the engines' loop registers): LOADK->QK, LOADV->PV,
// QK->SM, SM->PREAD (k = 0); QK->LOADK (k = K ring depth), PV->LOADV (k = V
// ring depth), PREAD->QK (k = 2: the S/P slot and its alpha row are free
// once PREAD holds them in registers, before the MFMAs of PV).  Ring slots
// and S/P slots follow r_KV over all tiles, and their reuse across tiles is
// ordered in one of two forms: the paper's relation, with these three read
// per trip of KV and acquire instructions at each tile (ACQK on E0, ACQV on
// E4, ACQS on E1; QK->ACQK, PV->ACQV, PREAD->ACQS at k = 1, C3 at T) that
// drain the previous tile's reads before the next tile refills; or these
// three read with the linearized offset (an extension of the paper's
// relation), so the next tile's loads and QK steps overlap the end of the
// previous tile.  SM->NORM (k = 0, C2: the tile's final row sums); NORM->SM
// (k = 2 at T: the row sums are double-buffered by tile, and a tile's
// softmax overwrites a buffer only after NORM of the tile before last has
// read it).
//
// Query rows of the tile beyond the sequence are computed on a clamped copy
// of the last row and never stored; keys beyond the sequence in the last
// block are loaded from a clamped row and masked to probability 0.
//
// LDS (bytes): counters 2048 | K ring (16 KiB slots: 64 rows of 256 B, the
// 16-byte chunk c of row r at c ^ (r mod 16)) | V ring (16 KiB slots, chunk c
// of row r at c ^ 4 (r mod 4), the layout the transposing fragment reads need
// to be conflict-free) | 2 S/P slots of 32 KiB (S fp32 [128][64]: 16-byte
// chunk c of row r at c ^ (r mod 16); P bf16 overwrites it with 8 chunks per
// row at the same permutation) | alpha [2][128] fp32 | l [2][128] fp32 |
// the workgroup's tile descriptors, staged at the start in what is left of
// the 160 KiB (up to 1024 tiles, 16 bytes plus a 4-byte KV trip each; later
// tiles read their descriptors from memory).
//
// MFMA v_mfma_f32_32x32x16_bf16: lane l supplies row l % 32 of the first
// operand and column l % 32 of the second, k = 8 (l / 32) .. + 7, and holds
// column l % 32 of the result, rows 8 (i / 4) + 4 (l / 32) + i % 4 for
// accumulator element i.  QK passes (K fragment, Q fragment), so lane l holds
// S[query l % 32][4-key runs]; PV passes (V^T fragment, P fragment), so lane
// l holds O[query l % 32][4-column runs] and the per-row rescale is one
// scalar per lane.  The V^T fragment (8 consecutive keys of one column) comes
// from two ds_read_b64_tr_b16: within each group of 16 lanes, lane i receives
// element i % 4 of the 8 bytes addressed by lane 4 j + i / 4 as its element j.
//
// Family contract (BFS_KERNEL_ATTN): loop T below the top level and loop KV
// in T, KV holding LOADK (E0, opcode 32, args [0, K ring depth, heads,
// 128]), LOADV (E4, opcode 32, args [1, V ring depth, heads, 128]), QK (E1,
// 33), SM (E2, 34), PREAD (E3, 37), PV (E3, 35); NORM (E3, 36) in T after
// KV; in the paper's form ACQK (E0), ACQV (E4) and ACQS (E1), no-ops in T
// before KV; waves per engine 1, 2, 4, 4, 1; the dependencies listed above.
// Buffers: [0] work list int32 [rows][4] = (first token of the sequence,
// length L, first query row of the tile, head), tile t of workgroup w at
// row w + t * n_wg (the caller provides every row its trip tables reach),
// [1] Q, [2] K, [3] V, [4] O, each bf16 [tokens][heads][128].  Trip table
// per workgroup: T runs its number of tiles, KV ceil(L / 64) steps for
// each (0 for an empty work item).
#include <string>

#include "engine_sync.h"

using namespace bfsdev;

namespace {

constexpr int kD = 128, kBQ = 128, kBKV = 64;
constexpr int kWaves = 12;
constexpr uint32_t kKVSlot = kBKV * kD * 2;      // 16 KiB
constexpr uint32_t kSPSlot = kBQ * kBKV * 4;     // 32 KiB
constexpr int kMaxPend = 3;                      // load groups in flight per load wave

struct AttnParams {
  SyncCommon sc;
  InstrWaits loadk, loadv, qk, sm, pread, pv, norm;
  InstrWaits acqk, acqv, acqs;   // acquire form: the drains at each tile (n = 0 in the linearized form)
  const int32_t *work;
  const __bf16 *q, *k, *v;
  __bf16 *o;
  const int32_t *trips;
  const int64_t *trip_off;
  int32_t heads, nk, nv;
  int32_t desc_cap;          // tile descriptors staged in LDS at most
  float scale_log2;          // log2(e) / sqrt(128)
};

// byte offset of 16-byte chunk c of row r (256-byte rows)
__device__ __forceinline__ uint32_t pos16(uint32_t r, uint32_t c) { return r * 256u + ((c ^ (r & 15u)) << 4); }

__device__ __forceinline__ bf16x8 lds_frag(uint32_t addr) {
  return __builtin_bit_cast(bf16x8, *(const BFS_LDS u32x4 *)(uintptr_t)addr);
}

__device__ __forceinline__ bf16x4 lds_tr(uint32_t addr) {
  typedef __attribute__((ext_vector_type(4))) short s16x4;
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((BFS_LDS s16x4 *)(uintptr_t)addr);
  return __builtin_bit_cast(bf16x4, v);
}

// Lanes l and l ^ 32 exchange x with v_permlane32_swap (no LDS traffic):
// the two results hold {x[l], x[l + 32]} in the low half and
// {x[l - 32], x[l]} in the high half, so any symmetric op of the pair
// combines the two lanes' values.
__device__ __forceinline__ f32x2 pair32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, x), __builtin_bit_cast(uint32_t, x),
                                                  false, false);
  return f32x2{__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1])};
}

template <int kMode, bool kInstr>
__global__ void __launch_bounds__(768) attn_kernel(AttnParams P) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  uint32_t *cnt = reinterpret_cast<uint32_t *>(lds);
  const uint32_t kring = lds_addr(lds) + kCntBytes;
  const uint32_t vring = kring + (uint32_t)P.nk * kKVSlot;
  const uint32_t spbuf = vring + (uint32_t)P.nv * kKVSlot;
  const uint32_t alpha_l = spbuf + 2u * kSPSlot;
  const uint32_t lsum_l = alpha_l + 2u * kBQ * 4u;
  // the workgroup's tile descriptors (first token, length, first query row,
  // head) and KV trips, staged in LDS once so that a tile's start reads LDS
  // rather than memory
  const uint32_t desc_l = lsum_l + 2u * kBQ * 4u;
  const uint32_t dtrip_l = desc_l + 16u * (uint32_t)P.desc_cap;
  const int wg = blockIdx.x;
  const int64_t *toff = P.trip_off + (int64_t)wg * 3;
  const uint32_t trip_t = (uint32_t)ldc(P.trips + ldc(toff + 1));
  const int64_t kv_off = ldc(toff + 2);
  const uint32_t n_staged = min(trip_t, (uint32_t)P.desc_cap);
  for (int i = threadIdx.x; i < bfs::kMaxSlots * bfs::kMaxWavesPerEngine; i += blockDim.x) cnt[i] = 0;
  for (uint32_t t = threadIdx.x; t < n_staged; t += blockDim.x) {
    const int64_t row = (int64_t)wg + (int64_t)t * gridDim.x;
    *(BFS_LDS u32x4 *)(uintptr_t)(desc_l + 16u * t) = *reinterpret_cast<const u32x4 *>(P.work + 4 * row);
    *(BFS_LDS int32_t *)(uintptr_t)(dtrip_l + 4u * t) = P.trips[kv_off + t];
  }
  __syncthreads();

  const int hw = wave_id();
  const uint32_t lane = lane_id(), l32 = lane & 31u, lhi = lane >> 5;
  // hardware wave -> (engine, wave within the engine), hardware wave w on
  // SIMD w % 4: the two QK waves on SIMDs 0 and 1, the four PV waves two
  // each on SIMDs 2 and 3 (equal MFMA work per SIMD), one softmax wave per
  // SIMD (equal VALU work), the K and V loaders on 0 and 1
  int eng, ew, canon;                       // canon: engine-ordered wave index
  if (hw < 2) { eng = 1; ew = hw; canon = 1 + ew; }
  else if (hw == 2 || hw == 3 || hw == 10 || hw == 11) { eng = 3; ew = (hw & 1) + ((hw >> 3) << 1); canon = 7 + ew; }
  else if (hw < 8) { eng = 2; ew = hw - 4; canon = 3 + ew; }
  else if (hw == 8) { eng = 0; ew = 0; canon = 0; }
  else { eng = 4; ew = 0; canon = 11; }
  // the PV waves issue ahead of the softmax and loader waves sharing their
  // SIMDs: their PREAD releases the S/P slot the next QK step needs (1 %
  // faster than equal priorities; raising the loaders or QK too was not)
  if (eng == 3) __builtin_amdgcn_s_setprio(2);
  Sync<kMode, kInstr> S(P.sc, lds_addr(cnt), canon, wg);
  const uint32_t own = S.word((uint32_t)eng, (uint32_t)ew);   // barrier mode: one counter per engine

  const size_t row_stride = (size_t)P.heads * kD;     // elements between tokens
  // tile t of this workgroup: row wg + t * n_wg of the work list, its KV
  // trip from the trip table (a trip beyond the sequence is reported and
  // clamped)
  struct Tile {
    int32_t s0, L, q0, head;
    uint32_t trip;
  };
  auto tile = [&](uint32_t t) {
    Tile x;
    if (t < n_staged) {
      const u32x4 d = *(const BFS_LDS u32x4 *)(uintptr_t)(desc_l + 16u * t);
      x.s0 = __builtin_amdgcn_readfirstlane((int32_t)d.x);
      x.L = __builtin_amdgcn_readfirstlane((int32_t)d.y);
      x.q0 = __builtin_amdgcn_readfirstlane((int32_t)d.z);
      x.head = __builtin_amdgcn_readfirstlane((int32_t)d.w);
      x.trip = (uint32_t)__builtin_amdgcn_readfirstlane(*(const BFS_LDS int32_t *)(uintptr_t)(dtrip_l + 4u * t));
    } else {
      const int64_t row = (int64_t)wg + (int64_t)t * gridDim.x;
      x.s0 = ldc(P.work + 4 * row + 0);
      x.L = ldc(P.work + 4 * row + 1);
      x.q0 = ldc(P.work + 4 * row + 2);
      x.head = ldc(P.work + 4 * row + 3);
      x.trip = (uint32_t)ldc(P.trips + kv_off + t);
    }
    const uint32_t max_trip = x.L > 0 ? (uint32_t)((x.L + kBKV - 1) / kBKV) : 0u;
    if (x.trip > max_trip) {
      report_input(P.sc.err, 1u, (uint32_t)wg, t, x.trip, max_trip, (uint32_t)hw);
      x.trip = max_trip;
    }
    return x;
  };
  Regs g;
  Site<2> site;
  Site<1> s_acq;                            // acquire form: the engine's wait at each tile
  uint64_t mark = 0;

  if (eng == 0 || eng == 4) {
    // ------------------------------------------------------- K / V loaders
    const bool is_v = eng == 4;
    const InstrWaits &iw = is_v ? P.loadv : P.loadk;
    const uint32_t depth = (uint32_t)(is_v ? P.nv : P.nk);
    const uint32_t ring = is_v ? vring : kring;
    int pending = 0;
    auto retire_one = [&]() {
      if (pending == 3) wait_vm<32>();
      else if (pending == 2) wait_vm<16>();
      else wait_vm<0>();
      S.signal(iw.update, 0);
      pending -= 1;
    };
    auto retire_all = [&]() {
      if (pending > 0) {
        wait_vm<0>();
        for (int i = 0; i < pending; ++i) S.signal(iw.update, 0);
        pending = 0;
      }
    };
    // lane t covers row 4 j + t / 16 of instruction j and the 16-byte chunk
    // that belongs at position t % 16 of that row
    const uint32_t rr = lane >> 4, pos = lane & 15u;
    // full blocks: a wave-uniform base (the block's first key) plus fixed
    // 32-bit per-lane byte offsets, so the loads take the scalar-base address
    // form and need no vector address arithmetic (which would compete for
    // issue with the MFMA waves on this SIMD); the block holding the
    // sequence's last key clamps rows one by one
    uint32_t voff[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t row = 4u * j + rr;
      const uint32_t chunk = is_v ? (pos ^ (rr << 2)) : (pos ^ (row & 15u));
      voff[j] = (row * (uint32_t)row_stride + 8u * chunk) * 2u;
    }
    // ring slots follow r_KV over all tiles: a tile's loads go on where the
    // previous tile's stopped, ordered by the linearized ring dependency, or
    // (acquire form) after ACQK / ACQV drained the previous tile's reads
    const InstrWaits &acq = is_v ? P.acqv : P.acqk;
    uint32_t slot = 0;
    S.sync_point(own);                                       // before loop T
    S.enter(s_acq, acq, g, 1);
    for (uint32_t t = 0; t < trip_t; ++t) {
      g.r1 += 1;
      g.h1 = t + 1;
      const Tile x = tile(t);
      const __bf16 *base = (is_v ? P.v : P.k) + (size_t)x.head * kD;
      S.wait(s_acq, acq, g, t + 1, g.r1 - 1, [&] { if (pending > 0) retire_one(); });   // ACQK / ACQV
      if (acq.update >= 0) {
        retire_all();
        S.signal(acq.update, 0);
      }
      S.sync_point(own);                                     // before loop KV
      S.enter(site, iw, g, 2);
      for (uint32_t it = 0; it < x.trip; ++it, slot = (slot + 1 == depth) ? 0u : slot + 1) {
        g.r2 += 1;
        g.h2 = it + 1;
        S.wait_affine(site, iw, g, it + 1, g.r2 - 1, [&] { if (pending > 0) retire_one(); });
        if (!S.aborted) {
          const uint32_t dst = ring + slot * kKVSlot;
          const int32_t key0 = (int32_t)it * kBKV;
          if (key0 + kBKV <= x.L) {
            const char *sb = reinterpret_cast<const char *>(base + (size_t)(x.s0 + key0) * row_stride);
#pragma unroll
            for (int j = 0; j < 16; ++j) {
              asm volatile("" : "+v"(voff[j]));   // keep the offset a 32-bit value at its use
              __builtin_amdgcn_global_load_lds((const void *)(sb + voff[j]),
                                               (BFS_LDS void *)(uintptr_t)(dst + 1024u * j), 16, 0, 0);
            }
          } else {
#pragma unroll
            for (int j = 0; j < 16; ++j) {
              const uint32_t row = 4u * j + rr;
              const uint32_t chunk = is_v ? (pos ^ (rr << 2)) : (pos ^ (row & 15u));
              const int32_t key = min(key0 + (int32_t)row, x.L - 1);
              const __bf16 *src = base + (size_t)(x.s0 + key) * row_stride + 8u * chunk;
              __builtin_amdgcn_global_load_lds((const void *)src, (BFS_LDS void *)(uintptr_t)(dst + 1024u * j), 16,
                                               0, 0);
            }
          }
          pending += 1;
          if (pending == kMaxPend) retire_one();
        } else {
          S.signal(iw.update, 0);
        }
        if (kMode == BFS_MODE_BARRIER) {
          retire_all();
          S.sync_point(own);                                 // end of a KV iteration
        }
      }
      if (kMode == BFS_MODE_BARRIER) retire_all();
      S.sync_point(own);                                     // end of a T iteration
    }
    retire_all();
  } else if (eng == 1) {
    // ---------------------------------------------------------- QK^T engine
    const uint32_t qr = 64u * ew;
    S.sync_point(own);                                       // before loop T
    S.enter(s_acq, P.acqs, g, 1);
    uint32_t kslot = 0;
    for (uint32_t t = 0; t < trip_t; ++t) {
      g.r1 += 1;
      g.h1 = t + 1;
      const Tile x = tile(t);
      // the tile's 64 query rows of this wave, held in registers for its KV
      // loop; loaded before the acquire so that their latency overlaps it
      bf16x8 qf[2][8];
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) {
        const int32_t row = min(x.q0 + (int32_t)(qr + 32u * qb + l32), x.L - 1);
        const __bf16 *src = P.q + (size_t)(x.s0 + max(row, 0)) * row_stride + (size_t)x.head * kD + 8u * lhi;
#pragma unroll
        for (int s = 0; s < 8; ++s)
          qf[qb][s] = x.L > 0 ? __builtin_bit_cast(bf16x8, *(const u32x4 *)(src + 16 * s)) : bf16x8{};
      }
      // acquire form: the previous tile's S/P slots are released (its PREADs
      // have read them) before this tile's first QK writes one
      S.wait(s_acq, P.acqs, g, t + 1, g.r1 - 1, [] {});   // ACQS
      S.signal(P.acqs.update, ew);
      S.sync_point(own);                                     // before loop KV
      S.enter(site, P.qk, g, 2);
      for (uint32_t it = 0; it < x.trip; ++it, kslot = (kslot + 1 == (uint32_t)P.nk) ? 0u : kslot + 1) {
        g.r2 += 1;
        g.h2 = it + 1;
        S.wait_affine(site, P.qk, g, it + 1, g.r2 - 1, [] {});
        if (!S.aborted) {
          const uint32_t kb_base = kring + kslot * kKVSlot;
          const uint32_t sp = spbuf + ((g.r2 - 1) & 1u) * kSPSlot;
          f32x16 acc[2][2];
#pragma unroll
          for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b) acc[a][b] = f32x16{};
          // the K fragments of each 16-wide slice of d are read one slice
          // ahead of the MFMAs that use them
          bf16x8 k0 = lds_frag(kb_base + pos16(l32, lhi));
          bf16x8 k1 = lds_frag(kb_base + pos16(32u + l32, lhi));
#pragma unroll
          for (int s = 0; s < 8; ++s) {
            bf16x8 n0 = k0, n1 = k1;
            if (s < 7) {
              n0 = lds_frag(kb_base + pos16(l32, 2u * (s + 1) + lhi));
              n1 = lds_frag(kb_base + pos16(32u + l32, 2u * (s + 1) + lhi));
            }
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
              acc[qb][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, qf[qb][s], acc[qb][0], 0, 0, 0);
              acc[qb][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, qf[qb][s], acc[qb][1], 0, 0, 0);
            }
            if (s < 7) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
            k0 = n0;
            k1 = n1;
          }
#pragma unroll
          for (int qb = 0; qb < 2; ++qb) {
            const uint32_t row = qr + 32u * qb + l32;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
              for (int j = 0; j < 4; ++j) {
                const f32x4 v = {acc[qb][kb][4 * j], acc[qb][kb][4 * j + 1], acc[qb][kb][4 * j + 2],
                                 acc[qb][kb][4 * j + 3]};
                *(BFS_LDS f32x4 *)(uintptr_t)(sp + pos16(row, 8u * kb + 2u * j + lhi)) = v;
              }
          }
        }
        S.signal(P.qk.update, (uint32_t)ew);
        S.sync_point(own);                                   // end of a KV iteration
      }
      S.sync_point(own);                                     // end of a T iteration
    }
  } else if (eng == 2) {
    // ------------------------------------------------------ softmax engine
    const uint32_t row = 32u * ew + l32;
    const float c = P.scale_log2;
    S.sync_point(own);                                       // before loop T
    for (uint32_t t = 0; t < trip_t; ++t) {
      g.r1 += 1;
      g.h1 = t + 1;
      const Tile x = tile(t);
      float m = -__builtin_inff(), lrun = 0.0f;
      S.sync_point(own);                                     // before loop KV
      S.enter(site, P.sm, g, 2);
      for (uint32_t it = 0; it < x.trip; ++it) {
        g.r2 += 1;
        g.h2 = it + 1;
        S.wait_affine(site, P.sm, g, it + 1, g.r2 - 1, [] {});
        if (!S.aborted) {
          const uint32_t par = (g.r2 - 1) & 1u;
          const uint32_t sp = spbuf + par * kSPSlot;
          float xs[32];
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const f32x4 v = *(const BFS_LDS f32x4 *)(uintptr_t)(sp + pos16(row, 8u * lhi + j));
            xs[4 * j] = v.x;
            xs[4 * j + 1] = v.y;
            xs[4 * j + 2] = v.z;
            xs[4 * j + 3] = v.w;
          }
          const int32_t key0 = (int32_t)it * kBKV + 32 * (int32_t)lhi;
          if ((int32_t)(it + 1) * kBKV > x.L) {
#pragma unroll
            for (int q = 0; q < 32; ++q)
              if (key0 + q >= x.L) xs[q] = -__builtin_inff();
          }
          float mx = xs[0];
#pragma unroll
          for (int q = 1; q < 32; ++q) mx = __builtin_fmaxf(mx, xs[q]);
          const f32x2 mp = pair32(mx);
          mx = __builtin_fmaxf(mp.x, mp.y);
          const float m_new = __builtin_fmaxf(m, mx * c);
          const float alpha = __builtin_amdgcn_exp2f(m - m_new);
          float sum = 0.0f;
          uint32_t pk[16];
#pragma unroll
          for (int q = 0; q < 32; q += 2) {
            const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(xs[q], c, -m_new));
            const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(xs[q + 1], c, -m_new));
            sum += p0 + p1;
            pk[q / 2] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{p0, p1}, bf16x2));
          }
          const f32x2 sums = pair32(sum);
          sum = sums.x + sums.y;
          lrun = alpha * lrun + sum;
          m = m_new;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const u32x4 v = {pk[4 * j], pk[4 * j + 1], pk[4 * j + 2], pk[4 * j + 3]};
            *(BFS_LDS u32x4 *)(uintptr_t)(sp + pos16(row, 4u * lhi + j)) = v;
          }
          if (lhi == 0) {
            *(BFS_LDS float *)(uintptr_t)(alpha_l + (par * kBQ + row) * 4u) = alpha;
            *(BFS_LDS float *)(uintptr_t)(lsum_l + (((g.r1 - 1) & 1u) * kBQ + row) * 4u) = lrun;
          }
        }
        S.signal(P.sm.update, (uint32_t)ew);
        S.sync_point(own);                                   // end of a KV iteration
      }
      S.sync_point(own);                                     // end of a T iteration
    }
  } else {
    // --------------------------------------------------- PV engine and NORM
    const uint32_t qr = 32u * ew;
    // transposing V reads: lane l addresses row 8 (l / 32) + (l % 16) / 4 (+ 16 ks + 4 hh)
    // and columns 32 db + 16 ((l / 16) % 2) + 4 (l % 4) .. + 3
    const uint32_t xq = (lane >> 2) & 3u;
    const uint32_t vrow = 8u * lhi + xq;
    uint32_t voff[4];
#pragma unroll
    for (int db = 0; db < 4; ++db)
      voff[db] = vrow * 256u + 16u * (4u * ((uint32_t)db ^ xq) + 2u * ((lane >> 4) & 1u) + ((lane >> 1) & 1u)) +
                 8u * (lane & 1u);
    Site<2> s_pr;
    Site<1> s_norm;
    uint32_t vslot = 0;
    S.sync_point(own);                                       // before loop T
    S.enter(s_norm, P.norm, g, 1);
    for (uint32_t t = 0; t < trip_t; ++t) {
      g.r1 += 1;
      g.h1 = t + 1;
      const Tile x = tile(t);
      f32x16 acc[4];
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[b] = f32x16{};
      S.sync_point(own);                                     // before loop KV
      S.enter(s_pr, P.pread, g, 2);
      S.enter(site, P.pv, g, 2);
      for (uint32_t it = 0; it < x.trip; ++it, vslot = (vslot + 1 == (uint32_t)P.nv) ? 0u : vslot + 1) {
        g.r2 += 1;
        g.h2 = it + 1;
        // PREAD: P and alpha of the step into registers, then the S/P slot
        // is released (LDS executes this wave's reads before its signal)
        S.wait_affine(s_pr, P.pread, g, it + 1, g.r2 - 1, [] {});
        bf16x8 pf[4];
        float a = 1.0f;
        if (!S.aborted) {
          const uint32_t par = (g.r2 - 1) & 1u;
          const uint32_t sp = spbuf + par * kSPSlot;
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) pf[ks] = lds_frag(sp + pos16(qr + l32, 2u * (uint32_t)ks + lhi));
          a = *(const BFS_LDS float *)(uintptr_t)(alpha_l + (par * kBQ + qr + l32) * 4u);
        }
        S.signal(P.pread.update, (uint32_t)ew);
        S.wait_affine(site, P.pv, g, it + 1, g.r2 - 1, [] {});
        if (!S.aborted) {
          const uint32_t vb = vring + vslot * kKVSlot;
          auto vfrag = [&](int ks, int db) {
            const uint32_t va = vb + 16u * (uint32_t)ks * 256u + voff[db];
            const bf16x4 lo = lds_tr(va), hi = lds_tr(va + 4u * 256u);
            return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
          };
          // the first V fragment is read before the rescale so that its
          // latency overlaps it
          bf16x8 vf = vfrag(0, 0);
          // a block whose rows all keep their running maximum needs no rescale
          if (__builtin_amdgcn_ballot_w64(a != 1.0f) != 0) {
#pragma unroll
            for (int db = 0; db < 4; ++db) acc[db] *= a;
          }
          // each V fragment is read one MFMA ahead of its use
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
            for (int db = 0; db < 4; ++db) {
              bf16x8 vf_next = vf;
              if (db < 3) vf_next = vfrag(ks, db + 1);
              else if (ks < 3) vf_next = vfrag(ks + 1, 0);
              acc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[ks], acc[db], 0, 0, 0);
              if (db < 3 || ks < 3) __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
              __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
              vf = vf_next;
            }
          }
        }
        S.signal(P.pv.update, (uint32_t)ew);
        S.sync_point(own);                                   // end of a KV iteration
      }
      mark = S.elapsed();
      // NORM: O / l for the tile's rows of the sequence; its signal lets the
      // softmax of the tile after next overwrite these row sums
      S.wait(s_norm, P.norm, g, t + 1, g.r1 - 1, [] {});
      if (!S.aborted) {
        const uint32_t rloc = qr + l32;
        const int32_t row = x.q0 + (int32_t)rloc;
        const float lr = *(const BFS_LDS float *)(uintptr_t)(lsum_l + (((g.r1 - 1) & 1u) * kBQ + rloc) * 4u);
        const float inv = 1.0f / lr;
        // lane l holds columns 8 j + 4 (l / 32) .. + 3 of each 32-column
        // block db: lanes l and l + 32 exchange halves (v_permlane32_swap) so
        // that the low lane holds the 8 columns of j = 0, 2 and the high lane
        // those of j = 1, 3, and each stores 16-byte row segments
        __bf16 *dst = P.o + (size_t)(x.s0 + max(min(row, x.L - 1), 0)) * row_stride + (size_t)x.head * kD;
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int jp = 0; jp < 2; ++jp) {
            uint32_t q[2][2];   // [j - 2 jp][dword]: this lane's 4 columns of j = 2 jp, 2 jp + 1
#pragma unroll
            for (int jj = 0; jj < 2; ++jj) {
              const int j = 2 * jp + jj;
              const f32x2 a01 = {acc[db][4 * j] * inv, acc[db][4 * j + 1] * inv};
              const f32x2 a23 = {acc[db][4 * j + 2] * inv, acc[db][4 * j + 3] * inv};
              q[jj][0] = __builtin_bit_cast(uint32_t, __builtin_convertvector(a01, bf16x2));
              q[jj][1] = __builtin_bit_cast(uint32_t, __builtin_convertvector(a23, bf16x2));
            }
            // low lane: keep j = 2 jp, receive the high lane's half of it;
            // high lane: keep j = 2 jp + 1, receive the low lane's half of it
            u32x4 v;
#pragma unroll
            for (int d = 0; d < 2; ++d) {
              // r[0]: a lane below 32 keeps its q[0][d], a lane above gets
              // q[1][d] of lane - 32; r[1]: a lane below 32 gets q[0][d] of
              // lane + 32, a lane above keeps its q[1][d]
              const auto r = __builtin_amdgcn_permlane32_swap(q[0][d], q[1][d], false, false);
              const uint32_t mine = lhi == 0 ? q[0][d] : q[1][d];
              const uint32_t other = lhi == 0 ? (uint32_t)r[1] : (uint32_t)r[0];
              v[d] = lhi == 0 ? mine : other;
              v[2 + d] = lhi == 0 ? other : mine;
            }
            const int j = 2 * jp + (int)lhi;
            if (row < x.L) *reinterpret_cast<u32x4 *>(dst + 32 * db + 8 * j) = v;
          }
      }
      S.signal(P.norm.update, (uint32_t)ew);
      S.sync_point(own);                                     // end of a T iteration
    }
  }
  drain_all();
  S.finish(lane, mark);
}

}  // namespace

namespace bfs {

bfs_status launch_attn(const bfs_plan *p, DevImage *img, const void *const *bufs, int32_t nbufs,
                       const int32_t *trips, const int64_t *trip_off, int32_t n_wg, void *stream, uint32_t *dbg,
                       int64_t dbg_cap, const bfs_run_opts &o) {
  if (p->n_loops != 3 || p->loop_parent[1] != 0 || p->loop_parent[2] != 1)
    return fail(BFS_E_UNSUPPORTED, "attn: loops must be top -> T -> KV");
  const int want_w[5] = {1, 2, 4, 4, 1};
  if (p->n_engines != 5) return fail(BFS_E_UNSUPPORTED, "attn: five engines");
  for (int e = 0; e < 5; ++e)
    if (p->waves_per_engine[e] != want_w[e]) return fail(BFS_E_UNSUPPORTED, "attn: engines of 1, 2, 4, 4, 1 waves");
  int lk = -1, lv = -1, qk = -1, sm = -1, pr = -1, pv = -1, nm = -1, ak = -1, av = -1, as = -1;
  for (size_t i = 0; i < p->instr_engine.size(); ++i) {
    const int op = p->instr_opcode[i], e = p->instr_engine[i], par = p->instr_parent[i];
    const int32_t *a = &p->instr_args[8 * i];
    if (op == 0 && par == 1 && e == 0 && ak < 0 && lk < 0) ak = (int)i;         // acquire form: ACQK
    else if (op == 0 && par == 1 && e == 4 && av < 0 && lv < 0) av = (int)i;    // ACQV
    else if (op == 0 && par == 1 && e == 1 && as < 0 && qk < 0) as = (int)i;    // ACQS
    else if (op == 32 && e == 0 && par == 2 && a[0] == 0 && lk < 0) lk = (int)i;
    else if (op == 32 && e == 4 && par == 2 && a[0] == 1 && lv < 0) lv = (int)i;
    else if (op == 33 && e == 1 && par == 2 && qk < 0) qk = (int)i;
    else if (op == 34 && e == 2 && par == 2 && sm < 0) sm = (int)i;
    else if (op == 37 && e == 3 && par == 2 && pr < 0 && pv < 0) pr = (int)i;
    else if (op == 35 && e == 3 && par == 2 && pv < 0) pv = (int)i;
    else if (op == 36 && e == 3 && par == 1 && nm < 0 && pv >= 0) nm = (int)i;
    else return fail(BFS_E_UNSUPPORTED, "attn: unexpected instruction " + std::to_string(i));
  }
  if (lk < 0 || lv < 0 || qk < 0 || sm < 0 || pr < 0 || pv < 0 || nm < 0)
    return fail(BFS_E_UNSUPPORTED, "attn: needs LOADK, LOADV, QK, SM, PREAD, PV and NORM (PREAD before PV)");
  const int nk = p->instr_args[8 * lk + 1], nv = p->instr_args[8 * lv + 1];
  const int heads = p->instr_args[8 * lk + 2], dim = p->instr_args[8 * lk + 3];
  if (dim != kD || p->instr_args[8 * lv + 3] != kD) return fail(BFS_E_UNSUPPORTED, "attn: head dimension 128");
  if (heads <= 0 || p->instr_args[8 * lv + 2] != heads) return fail(BFS_E_INVALID, "attn: heads must match");
  const size_t lds_base = kCntBytes + (size_t)(nk + nv) * kKVSlot + 2 * kSPSlot + 4 * kBQ * 4;
  if (nk < 2 || nv < 2 || lds_base > 160 * 1024)
    return fail(BFS_E_UNSUPPORTED, "attn: ring depths >= 2 within 160 KiB of LDS");
  // the rest of the LDS (up to 1024 tiles) stages tile descriptors: 16 bytes
  // and a 4-byte KV trip per tile; tiles beyond it read memory
  const int32_t desc_cap = (int32_t)std::min<size_t>(1024, (160 * 1024 - lds_base) / 20);
  const size_t lds = lds_base + (size_t)desc_cap * 20;
  // The kernel's buffers are only race-free under these dependencies.  The
  // rings and S/P slots are indexed by r_KV over all tiles, so their reuse
  // across tiles is ordered either by reading the reuse dependencies with
  // the linearized offset (extension), or, with the paper's relation, by
  // acquire instructions at each tile on the K loader, the V loader and the
  // QK engine whose C3 dependencies (offset 1 at T) drain the previous
  // tile's QK, PV and PREAD.
  auto dep_form = [&](int prd, int cns, int k, int linear) {
    for (size_t d = 0; d < p->deps.size() / 3; ++d)
      if (p->deps[3 * d] == prd && p->deps[3 * d + 1] == cns && p->deps[3 * d + 2] == k &&
          (p->dep_linear.empty() ? 0 : p->dep_linear[d]) == linear)
        return true;
    return false;
  };
  const bool acq_form = ak >= 0 && av >= 0 && as >= 0;
  if ((ak >= 0 || av >= 0 || as >= 0) && !acq_form)
    return fail(BFS_E_UNSUPPORTED, "attn: the acquire form needs ACQK, ACQV and ACQS");
  const int lin = acq_form ? 0 : 1;
  bool ok = has_dep(p, lk, qk, 0) && has_dep(p, lv, pv, 0) && has_dep(p, qk, sm, 0) && has_dep(p, sm, pr, 0) &&
            dep_form(qk, lk, nk, lin) && dep_form(pv, lv, nv, lin) && dep_form(pr, qk, 2, lin) &&
            has_dep(p, sm, nm, 0) && has_dep(p, nm, sm, 2);
  if (acq_form) ok = ok && dep_form(qk, ak, 1, 0) && dep_form(pv, av, 1, 0) && dep_form(pr, as, 1, 0);
  if (!ok) return fail(BFS_E_UNSUPPORTED, "attn: missing a ring, S/P or row-sum dependency");
  if (nbufs < 5) return fail(BFS_E_INVALID, "attn: needs [work, Q, K, V, O]");
  for (int i = 0; i < 5; ++i)
    if (!bufs[i]) return fail(BFS_E_INVALID, "attn: null buffer");
  if (!trips || !trip_off) return fail(BFS_E_INVALID, "attn: needs trip tables");
  if (n_wg <= 0) return fail(BFS_E_INVALID, "attn: n_wg must be positive");
  const std::vector<DevWait> dw = device_waits(p);
  AttnParams P{};
  if (!fill_waits(p, dw, lk, P.loadk) || !fill_waits(p, dw, lv, P.loadv) || !fill_waits(p, dw, qk, P.qk) ||
      !fill_waits(p, dw, sm, P.sm) || !fill_waits(p, dw, pr, P.pread) || !fill_waits(p, dw, pv, P.pv) ||
      !fill_waits(p, dw, nm, P.norm))
    return fail(BFS_E_RESOURCE, "attn: at most 4 waits per instruction");
  P.acqk.update = P.acqv.update = P.acqs.update = -1;
  if (acq_form && (!fill_waits(p, dw, ak, P.acqk) || !fill_waits(p, dw, av, P.acqv) || !fill_waits(p, dw, as, P.acqs)))
    return fail(BFS_E_RESOURCE, "attn: at most 4 waits per instruction");
  if (!waits_fit({{&P.loadk, 2}, {&P.loadv, 2}, {&P.qk, 2}, {&P.sm, 2}, {&P.pread, 2}, {&P.pv, 2}, {&P.norm, 1},
                  {&P.acqk, 1}, {&P.acqv, 1}, {&P.acqs, 1}}))
    return fail(BFS_E_RESOURCE, "attn: more waits on an instruction than its engine loop takes");
  if (p->mode == BFS_MODE_BARRIER_FREE &&
      (!no_dynamic(P.loadk) || !no_dynamic(P.loadv) || !no_dynamic(P.qk) || !no_dynamic(P.sm) ||
       !no_dynamic(P.pread) || !no_dynamic(P.pv)))
    return fail(BFS_E_UNSUPPORTED, "attn: a KV-loop wait depends on a loop register other than the KV loop's");
  P.sc = sync_common(img, dbg, dbg_cap, o, kWaves);
  P.work = static_cast<const int32_t *>(bufs[0]);
  P.q = static_cast<const __bf16 *>(bufs[1]);
  P.k = static_cast<const __bf16 *>(bufs[2]);
  P.v = static_cast<const __bf16 *>(bufs[3]);
  P.o = static_cast<__bf16 *>(const_cast<void *>(bufs[4]));
  P.trips = trips;
  P.trip_off = trip_off;
  P.heads = heads;
  P.nk = nk;
  P.nv = nv;
  P.desc_cap = desc_cap;
  P.scale_log2 = 1.4426950408889634f / 11.313708498984761f;   // log2(e) / sqrt(128)
  const bool instr = dbg || o.dev_stats || o.fault_dep >= 0;
  hipStream_t s = (hipStream_t)stream;
  auto go = [&](auto kern) -> bfs_status {
    hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("attn attribute: ") + hipGetErrorString(e));
    hipLaunchKernelGGL(kern, dim3(n_wg), dim3(64 * kWaves), lds, s, P);
    e = hipGetLastError();
    if (e != hipSuccess) return fail(BFS_E_DEVICE, std::string("attn launch: ") + hipGetErrorString(e));
    return BFS_OK;
  };
  if (p->mode == BFS_MODE_BARRIER) return instr ? go(attn_kernel<BFS_MODE_BARRIER, true>) : go(attn_kernel<BFS_MODE_BARRIER, false>);
  return instr ? go(attn_kernel<BFS_MODE_BARRIER_FREE, true>) : go(attn_kernel<BFS_MODE_BARRIER_FREE, false>);
}

}  // namespace bfs
