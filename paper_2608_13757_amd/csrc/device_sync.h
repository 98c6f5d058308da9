// Device-side synchronization primitives for gfx950 engine wavefronts.
//
// A semaphore of the paper (Section 3.3: wait until the counter reaches a
// threshold, increment at retirement) is a 32-bit LDS word.  A wait polls the
// word with a plain LDS read and sleeps between polls; a retirement is an LDS
// atomic add issued only after the instruction's memory effects are complete
// (s_waitcnt), in the engine's program order.  The poll and the add are
// written as inline assembly so that the compiler does not insert a
// conservative "vmcnt(0)" before them: a load engine keeps several
// direct-to-LDS loads in flight and retires them one by one with counted
// waits.
//
// Barrier mode (Section 3.4): drain every outstanding memory operation, meet
// at the workgroup barrier, reset the wave's own counter words, meet again.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define BFS_LDS __attribute__((address_space(3)))

namespace bfsdev {

__device__ __forceinline__ uint32_t lane_id() { return __lane_id(); }

__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
}

__device__ __forceinline__ uint32_t uniform(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }

// 32-bit LDS address of a __shared__ object.
template <typename T>
__device__ __forceinline__ uint32_t lds_addr(T *p) {
  return (uint32_t)(uintptr_t)(BFS_LDS void *)(p);
}

// Load through the constant address space: with a wave-uniform address this
// is a scalar load, tracked by lgkmcnt instead of vmcnt, so it never forces a
// wait on outstanding vector-memory (direct-to-LDS) loads.
template <typename T>
__device__ __forceinline__ T ldc(const T *p) {
  return *(const __attribute__((address_space(4))) T *)(p);
}

// A struct of int32 fields, loaded field by field through ldc.
template <typename T>
__device__ __forceinline__ T ldc_struct(const T *p) {
  static_assert(sizeof(T) % 4 == 0, "int32 fields");
  T out;
  const int32_t *src = reinterpret_cast<const int32_t *>(p);
  int32_t *dst = reinterpret_cast<int32_t *>(&out);
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 4); ++i) dst[i] = ldc(src + i);
  return out;
}

// One LDS read of a counter word, completed before returning.
__device__ __forceinline__ uint32_t lds_poll(uint32_t addr) {
  uint32_t v;
  asm volatile("ds_read_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(addr) : "memory");
  return v;
}

// Increment a counter word by n: the add is issued with only lane 0 active
// (the exec mask is saved and restored around it).
__device__ __forceinline__ void lds_add(uint32_t addr, uint32_t n) {
  uint64_t saved;
  asm volatile(
      "s_mov_b64 %0, exec\n\t"
      "s_mov_b64 exec, 1\n\t"
      "ds_add_u32 %1, %2\n\t"
      "s_mov_b64 exec, %0"
      : "=&s"(saved)
      : "v"(addr), "v"(n)
      : "memory");
}

__device__ __forceinline__ void lds_store(uint32_t addr, uint32_t v) {
  if (lane_id() == 0) asm volatile("ds_write_b32 %0, %1" ::"v"(addr), "v"(v) : "memory");
}

// Complete every outstanding memory operation of this wave, then retire:
// the counter add is ordered after all of them.
__device__ __forceinline__ void retire_all_and_add(uint32_t addr, uint32_t n) {
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
  lds_add(addr, n);
}

__device__ __forceinline__ void drain_all() { asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory"); }

// Counted wait on vector-memory operations (direct-to-LDS loads complete in
// issue order): at most N may remain outstanding.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Runtime-count vector-memory wait (n <= 15).
__device__ __forceinline__ void wait_vm_dyn(int n) {
  switch (n) {
    case 0: wait_vm<0>(); break;
    case 1: wait_vm<1>(); break;
    case 2: wait_vm<2>(); break;
    case 3: wait_vm<3>(); break;
    case 4: wait_vm<4>(); break;
    case 5: wait_vm<5>(); break;
    case 6: wait_vm<6>(); break;
    case 7: wait_vm<7>(); break;
    case 8: wait_vm<8>(); break;
    case 9: wait_vm<9>(); break;
    case 10: wait_vm<10>(); break;
    case 11: wait_vm<11>(); break;
    case 12: wait_vm<12>(); break;
    case 13: wait_vm<13>(); break;
    case 14: wait_vm<14>(); break;
    default: wait_vm<15>(); break;
  }
}

// Wait until at most n vector-memory operations are outstanding, rounding n
// down to a value the wait instruction encodes (waiting for more is safe).
__device__ __forceinline__ void wait_vm_atmost(uint32_t n) {
  if (n >= 48) wait_vm<48>();
  else if (n >= 32) wait_vm<32>();
  else if (n >= 16) wait_vm<16>();
  else if (n >= 8) wait_vm<8>();
  else if (n >= 4) wait_vm<4>();
  else if (n >= 2) wait_vm<2>();
  else if (n >= 1) wait_vm<1>();
  else wait_vm<0>();
}

// Only LDS operations completed (the engine's own LDS reads and writes).
__device__ __forceinline__ void drain_lds() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// 100 MHz wall clock.
__device__ __forceinline__ uint64_t now_ticks() { return __builtin_amdgcn_s_memrealtime(); }

// Per-wave timing counters (opt-in; see bfs_run_opts.dev_stats).
struct WaveStats {
  uint64_t t_start = 0, blocked = 0, n_blocked = 0, barrier = 0, own_loads = 0, polls = 0;
  bool on = false;
};

// Outcome of one wait, for the debug log.
struct WaitResult {
  uint32_t observed;
  bool ok;
};

// Poll the counter words of the nw producer waves (consecutive words from
// addr) until every one is >= thr.  Gives up after max_polls polls.
// Minimum of v over lanes 0 .. nw - 1, read lane by lane into scalar
// registers (no cross-lane LDS traffic; nw is at most kMaxWavesPerEngine).
__device__ __forceinline__ uint32_t lane_min(uint32_t v, int nw) {
  uint32_t m = 0xffffffffu;
  for (int i = 0; i < nw; ++i) m = min(m, (uint32_t)__builtin_amdgcn_readlane((int)v, i));
  return m;
}

__device__ __forceinline__ WaitResult wait_geq(uint32_t addr, int nw, uint32_t thr, uint64_t max_polls) {
  WaitResult r{0, true};
  if (thr == 0) return r;
  const uint32_t lane = lane_id();
  const uint32_t a = addr + 4u * (lane < (uint32_t)nw ? lane : 0u);
  const uint64_t want = (nw >= 64) ? ~0ull : ((1ull << nw) - 1ull);
  uint64_t polls = 0;
  while (true) {
    uint32_t v = lds_poll(a);
    uint64_t good = __ballot(v >= thr) & want;
    if (good == want) {
      r.observed = lane_min(v, nw);      // minimum over the producer waves
      return r;
    }
    if (++polls > max_polls) {
      r.observed = lane_min(v, nw);
      r.ok = false;
      return r;
    }
    __builtin_amdgcn_s_sleep(1);
  }
}

// Poll one counter word until it reaches thr, sleeping between polls.  The
// loop body is a handful of scalar instructions, so a blocked wave takes few
// issue slots from the working waves of its compute unit.  Returns the last
// value seen; ok = false when max_polls polls did not suffice.
// Poll one counter word until it reaches thr.  max_polls is clamped to 32
// bits so the poll count stays a scalar 32-bit value (a 64-bit count is
// compared with vector instructions).
__device__ __forceinline__ WaitResult spin_geq(uint32_t addr, uint32_t thr, uint64_t max_polls) {
  const uint32_t limit = max_polls > 0xffffffffull ? 0xffffffffu : (uint32_t)max_polls;
  uint32_t polls = 0;
  while (true) {
    const uint32_t v = uniform(lds_poll(addr));
    if (v >= thr) return WaitResult{v, true};
    if (++polls > limit) return WaitResult{v, false};
    // back off: 64 clocks between the first polls, then 256
    if (polls < 8) __builtin_amdgcn_s_sleep(1);
    else __builtin_amdgcn_s_sleep(4);
  }
}

// Threshold of Eq. 5 from the consumer engine's loop registers.
__device__ __forceinline__ uint32_t eq5(uint32_t r_P, uint32_t rhat_S, int k, int sub, int N, int K, int mask) {
  if (mask && !(rhat_S > (uint32_t)k)) return 0u;
  int v = N * ((int)r_P - sub) - (N - K);
  return v > 0 ? (uint32_t)v : 0u;
}

// Barrier-mode synchronization point: drain, handshake, reset own counter
// words, handshake.
__device__ __forceinline__ void region_sync(uint32_t own_words, int n_words) {
  drain_all();
  __builtin_amdgcn_s_barrier();
  if (lane_id() < (uint32_t)n_words)
    asm volatile("ds_write_b32 %0, %1\n\ts_waitcnt lgkmcnt(0)" ::"v"(own_words + 4u * lane_id()), "v"(0u) : "memory");
  __builtin_amdgcn_s_barrier();
}

// Error word layout: [0] code, then six code-specific words.
//   code 1 (a wait gave up): [1] dep, [2] wg, [3] instance, [4] threshold,
//          [5] observed, [6] wave;
//   code 2 (a run-time input was rejected): [1] what (1 trip count beyond
//          the work item, 2 trip table disagrees with a static loop, 3 load
//          offset beyond 32 bits, 4 trip count beyond the ring-slot reuse the
//          program's dependencies order), [2] wg, [3] index, [4] value,
//          [5] limit, [6] wave.
// Branch-uniform on purpose: every lane tries the same compare-and-swap and
// a ballot tells the wave whether one of its lanes won, so no control flow
// here depends on the lane (a lane-dependent branch would make the callers'
// engine flags look divergent to the compiler).  The first error wins.
__device__ __forceinline__ void report_error(uint32_t *err, uint32_t code, uint32_t w1, uint32_t w2, uint32_t w3,
                                             uint32_t w4, uint32_t w5, uint32_t w6) {
  if (err == nullptr) return;
  const uint32_t old = atomicCAS(err, 0u, code);
  if (__ballot(old == 0u) != 0ull) {
    err[1] = w1;
    err[2] = w2;
    err[3] = w3;
    err[4] = w4;
    err[5] = w5;
    err[6] = w6;
  }
}

__device__ __forceinline__ void report_deadlock(uint32_t *err, uint32_t dep, uint32_t wg, uint32_t inst,
                                                uint32_t thr, uint32_t obs, uint32_t wave) {
  report_error(err, 1u, dep, wg, inst, thr, obs, wave);
}

__device__ __forceinline__ void report_input(uint32_t *err, uint32_t what, uint32_t wg, uint32_t index,
                                             uint32_t value, uint32_t limit, uint32_t wave) {
  report_error(err, 2u, what, wg, index, value, limit, wave);
}

// Debug log entry (dependency, consumer instance, threshold, observed).
__device__ __forceinline__ void log_wait(uint32_t *entries, int64_t cap, uint32_t &n, uint32_t dep, uint32_t inst,
                                         uint32_t thr, uint32_t obs) {
  if (entries && lane_id() == 0 && (int64_t)n < cap) {
    uint4 v = make_uint4(dep, inst, thr, obs);
    *reinterpret_cast<uint4 *>(entries + 4 * (int64_t)n) = v;
  }
  n += 1;
}

}  // namespace bfsdev
