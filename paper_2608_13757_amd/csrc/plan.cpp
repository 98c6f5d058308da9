// Host-side planner: validates a structured program and computes, for every
// dependency, the barrier-free wait of Sections 5.2-5.5 (or the barrier-mode
// static wait of Section 3.4).  Pure host code; needs no GPU.
#include <atomic>
#include <algorithm>
#include <cstring>
#include <map>
#include <string>
#include <vector>

#include "bfs_internal.h"

namespace bfs {

static thread_local std::string g_last_error;

void set_error(const std::string &msg) { g_last_error = msg; }

bfs_status fail(bfs_status s, const std::string &msg) {
  g_last_error = msg;
  return s;
}

namespace {

struct Pos {       // position of an instruction inside one loop body
  int32_t item;    // index of the body item holding it (its block or a child loop)
  int32_t sub;     // index inside the block when the item is its block, else -1
};

// Chain of loops from the top level down to l.
std::vector<int32_t> path_to(const bfs_plan &p, int32_t l) {
  std::vector<int32_t> v;
  for (int32_t x = l; x >= 0; x = p.loop_parent[x]) v.push_back(x);
  std::reverse(v.begin(), v.end());
  return v;
}

bfs_status validate_and_index(bfs_plan &p, std::vector<int32_t> &instr_block,
                              std::vector<int32_t> &instr_sub, std::vector<int32_t> &block_loop,
                              std::vector<int32_t> &block_item, std::vector<int32_t> &loop_item) {
  const int32_t L = p.n_loops, B = (int32_t)p.block_off.size() - 1, I = (int32_t)p.instr_engine.size();
  if (L < 1 || L > kMaxLoops) return fail(BFS_E_RESOURCE, "n_loops must be 1.." + std::to_string(kMaxLoops));
  if (p.n_engines < 1 || p.n_engines > kMaxEngines) return fail(BFS_E_INVALID, "n_engines must be 1..8");
  for (int e = 0; e < p.n_engines; ++e)
    if (p.waves_per_engine[e] < 1 || p.waves_per_engine[e] > kMaxWavesPerEngine)
      return fail(BFS_E_INVALID, "waves_per_engine must be 1..8");
  if (p.loop_parent[0] != -1) return fail(BFS_E_INVALID, "loop 0 must be the top level (parent -1)");
  if ((int32_t)p.body_off.size() != L + 1 || p.body_off[0] != 0)
    return fail(BFS_E_INVALID, "body_off must have n_loops + 1 entries starting at 0");
  for (int32_t l = 0; l < L; ++l)
    if (p.body_off[l + 1] < p.body_off[l]) return fail(BFS_E_INVALID, "body_off not monotone");
  if (p.block_off.empty() || p.block_off[0] != 0) return fail(BFS_E_INVALID, "block_off must start at 0");
  for (int32_t b = 0; b < B; ++b)
    if (p.block_off[b + 1] < p.block_off[b]) return fail(BFS_E_INVALID, "block_off not monotone");
  if ((int32_t)p.block_instrs.size() != p.block_off[B])
    return fail(BFS_E_INVALID, "block_instrs length does not match block_off");

  loop_item.assign(L, -1);
  block_loop.assign(B, -1);
  block_item.assign(B, -1);
  for (int32_t l = 0; l < L; ++l) {
    for (int32_t it = p.body_off[l]; it < p.body_off[l + 1]; ++it) {
      int32_t kind = p.body_kind[it], id = p.body_id[it];
      if (kind == 0) {
        if (id < 0 || id >= B) return fail(BFS_E_INVALID, "body references a bad block id");
        if (block_loop[id] != -1) return fail(BFS_E_INVALID, "block listed twice");
        block_loop[id] = l;
        block_item[id] = it - p.body_off[l];
      } else if (kind == 1) {
        if (id <= 0 || id >= L) return fail(BFS_E_INVALID, "body references a bad loop id");
        if (loop_item[id] != -1) return fail(BFS_E_INVALID, "loop listed twice");
        if (p.loop_parent[id] != l)
          return fail(BFS_E_INVALID, "loop " + std::to_string(id) + " listed outside its parent");
        loop_item[id] = it - p.body_off[l];
      } else {
        return fail(BFS_E_INVALID, "body_kind must be 0 (block) or 1 (loop)");
      }
    }
  }
  for (int32_t l = 1; l < L; ++l) {
    if (loop_item[l] == -1) return fail(BFS_E_INVALID, "loop " + std::to_string(l) + " not in any body");
    // parent chain must reach the top level without cycles
    int32_t x = l, steps = 0;
    while (x > 0 && steps <= L) { x = p.loop_parent[x]; ++steps; }
    if (x != 0) return fail(BFS_E_INVALID, "loop parents do not form a tree");
  }
  for (int32_t b = 0; b < B; ++b)
    if (block_loop[b] == -1) return fail(BFS_E_INVALID, "block " + std::to_string(b) + " not in any body");

  instr_block.assign(I, -1);
  instr_sub.assign(I, -1);
  for (int32_t b = 0; b < B; ++b)
    for (int32_t j = p.block_off[b]; j < p.block_off[b + 1]; ++j) {
      int32_t i = p.block_instrs[j];
      if (i < 0 || i >= I) return fail(BFS_E_INVALID, "block lists a bad instruction id");
      if (instr_block[i] != -1) return fail(BFS_E_INVALID, "instruction listed twice");
      instr_block[i] = b;
      instr_sub[i] = j - p.block_off[b];
    }
  for (int32_t i = 0; i < I; ++i) {
    if (instr_block[i] == -1) return fail(BFS_E_INVALID, "instruction " + std::to_string(i) + " in no block");
    if (p.instr_engine[i] < 0 || p.instr_engine[i] >= p.n_engines)
      return fail(BFS_E_INVALID, "instruction " + std::to_string(i) + " has a bad engine");
  }
  const int32_t D = (int32_t)p.deps.size() / 3;
  for (int32_t d = 0; d < D; ++d) {
    int32_t a = p.deps[3 * d], c = p.deps[3 * d + 1], k = p.deps[3 * d + 2];
    if (a < 0 || a >= I || c < 0 || c >= I || a == c || k < 0)
      return fail(BFS_E_INVALID, "dependency " + std::to_string(d) + " is malformed");
  }
  if (p.tile_elems < 0 || p.tile_elems > 256 || p.tile_elems % 64 != 0)
    return fail(BFS_E_INVALID, "tile_elems must be a multiple of 64 in [0, 256]");
  return BFS_OK;
}

}  // namespace

bfs_status plan_build(bfs_plan &p) {
  std::vector<int32_t> instr_block, instr_sub, block_loop, block_item, loop_item;
  bfs_status st = validate_and_index(p, instr_block, instr_sub, block_loop, block_item, loop_item);
  if (st != BFS_OK) return st;
  const int32_t L = p.n_loops, I = (int32_t)p.instr_engine.size(), D = (int32_t)p.deps.size() / 3;
  const int32_t E = p.n_engines;

  p.instr_parent.assign(I, -1);
  for (int32_t i = 0; i < I; ++i) p.instr_parent[i] = block_loop[instr_block[i]];
  p.loop_depth.assign(L, 0);
  for (int32_t l = 1; l < L; ++l) p.loop_depth[l] = (int32_t)path_to(p, l).size() - 1;

  // Position of instruction i in the body of its ancestor loop S.
  auto pos_in = [&](int32_t i, int32_t S) -> Pos {
    int32_t l = p.instr_parent[i];
    if (l == S) return Pos{block_item[instr_block[i]], instr_sub[i]};
    int32_t child = l;
    while (p.loop_parent[child] != S) child = p.loop_parent[child];
    return Pos{loop_item[child], -1};
  };
  auto lca = [&](int32_t a, int32_t b) {
    std::vector<int32_t> pa = path_to(p, a), pb = path_to(p, b);
    int32_t s = 0;
    for (size_t j = 0; j < pa.size() && j < pb.size() && pa[j] == pb[j]; ++j) s = pa[j];
    return s;
  };
  // Listing order of the instructions of engine e directly in loop l's body.
  auto direct_instrs = [&](int32_t l, int32_t e) {
    std::vector<int32_t> v;
    for (int32_t it = p.body_off[l]; it < p.body_off[l + 1]; ++it)
      if (p.body_kind[it] == 0) {
        int32_t b = p.body_id[it];
        for (int32_t j = p.block_off[b]; j < p.block_off[b + 1]; ++j)
          if (p.instr_engine[p.block_instrs[j]] == e) v.push_back(p.block_instrs[j]);
      }
    return v;
  };

  p.formulas.assign(D, bfs_formula{});
  p.static_waits.assign(D, bfs_static_wait{});
  std::map<std::pair<int32_t, int32_t>, int32_t> slot_of_loop_engine;  // per-loop allocation
  std::map<int32_t, int32_t> slot_of_instr;                            // per-instruction allocation
  std::map<int32_t, int32_t> slot_of_engine;                           // per-engine allocation
  p.fallback_loops = 0;
  for (int32_t d = 0; d < D; ++d) {
    const int32_t a = p.deps[3 * d], c = p.deps[3 * d + 1], k = p.deps[3 * d + 2];
    const int32_t P = p.instr_parent[a];
    const int32_t S = lca(P, p.instr_parent[c]);
    const Pos pa = pos_in(a, S), pc = pos_in(c, S);
    const bool forward = pa.item < pc.item || (pa.item == pc.item && pa.sub < pc.sub);
    const std::string tag = "dependency " + std::to_string(d) + " (" + std::to_string(a) + " -> " +
                            std::to_string(c) + ", offset " + std::to_string(k) + ")";
    bfs_formula f{};
    f.dep = d;
    f.loop_S = S;
    f.loop_P = P;
    f.k = k;
    f.prd_engine = p.instr_engine[a];
    f.cns_engine = p.instr_engine[c];
    f.forward = forward ? 1 : 0;
    if (p.dep_linear[d]) {                          // extension: offset over all trips of S
      if (P != S) return fail(BFS_E_NOT_ALLOCATABLE, tag + ": a linearized offset needs the producer directly in S");
      if (!forward && k == 0)
        return fail(BFS_E_ORDER, tag + ": offset 0 needs the producer before the consumer");
      f.kase = 6;
      f.expr_sub = k;
    } else if (P == S) {                            // C1: producer directly in S
      if (!forward && k == 0)
        return fail(BFS_E_ORDER, tag + ": offset 0 needs the producer before the consumer");
      f.kase = 1;
      f.expr_sub = k;
    } else if (forward && k == 0) {                 // C2: nested producer, forward
      f.kase = 2;
      f.expr_sub = 0;
    } else if (!forward && k == 1) {                // C3: nested producer, backward
      f.kase = 3;
      f.expr_sub = 0;
    } else if (!forward && k == 0) {
      return fail(BFS_E_ORDER, tag + ": nested backward producer at offset 0 is unsatisfiable");
    } else if (!(p.flags & BFS_PLAN_BARRIER_FALLBACK)) {
      return fail(BFS_E_NOT_ALLOCATABLE,
                  tag + (forward ? ": nested forward producer needs offset 0" : ": nested backward producer needs offset 1"));
    } else {                                        // Section 5.2 fallback: barriers at S's iteration ends
      f.kase = 4;
      f.expr_sub = 0;
    }
    f.needs_mask = (k > 0 && f.kase != 6) ? 1 : 0;
    if (f.kase == 4) {
      f.N = 0;
      f.K = 0;
      f.counter = -1;
      if (S != 0) p.fallback_loops |= 1u << S;
    } else if (p.alloc == BFS_ALLOC_PER_ENGINE) {
      // one counter per producer engine; the consumer keeps snapshots of the
      // producer engine's running count at the producer's position
      f.N = 0;
      f.K = 0;
      f.snap_slots = P == S ? k + 1 : 1;
      auto it = slot_of_engine.find(f.prd_engine);
      if (it == slot_of_engine.end()) it = slot_of_engine.emplace(f.prd_engine, (int32_t)slot_of_engine.size()).first;
      f.counter = it->second;
    } else if (p.alloc == BFS_ALLOC_PER_INSTR) {
      f.N = 1;
      f.K = 1;
      auto it = slot_of_instr.find(a);
      if (it == slot_of_instr.end()) it = slot_of_instr.emplace(a, (int32_t)slot_of_instr.size()).first;
      f.counter = it->second;
    } else {
      std::vector<int32_t> v = direct_instrs(P, f.prd_engine);
      f.N = (int32_t)v.size();
      f.K = (int32_t)(std::find(v.begin(), v.end(), a) - v.begin()) + 1;
      auto key = std::make_pair(P, f.prd_engine);
      auto it = slot_of_loop_engine.find(key);
      if (it == slot_of_loop_engine.end())
        it = slot_of_loop_engine.emplace(key, (int32_t)slot_of_loop_engine.size()).first;
      f.counter = it->second;
    }
    p.formulas[d] = f;

    // Barrier mode: same region iff offset 0, both directly in S, producer
    // first, and no loop statement between them in S's body.
    bfs_static_wait w{};
    w.dep = d;
    w.prd_engine = f.prd_engine;
    if (k == 0 && P == S && p.instr_parent[c] == S && forward) {
      bool separated = false;
      for (int32_t it = pa.item + 1; it < pc.item; ++it)
        if (p.body_kind[p.body_off[S] + it] == 1) separated = true;
      if (!separated) {
        int32_t seg = 0;   // first item of the producer's region
        for (int32_t it = pa.item - 1; it >= 0; --it)
          if (p.body_kind[p.body_off[S] + it] == 1) { seg = it + 1; break; }
        int32_t ord = 0;
        for (int32_t it = seg; it <= pa.item; ++it) {
          int32_t b = p.body_id[p.body_off[S] + it];
          for (int32_t j = p.block_off[b]; j < p.block_off[b + 1]; ++j) {
            int32_t ins = p.block_instrs[j];
            if (p.instr_engine[ins] == f.prd_engine) ++ord;
            if (ins == a) break;
          }
        }
        w.same_region = 1;
        w.ordinal = ord;
      }
    }
    p.static_waits[d] = w;
  }

  // Counters each instruction increments at retirement.
  p.instr_update.assign(I, -1);
  if (p.mode == BFS_MODE_BARRIER) {
    for (int32_t i = 0; i < I; ++i) p.instr_update[i] = p.instr_engine[i];
    p.n_counters = E;
  } else if (p.alloc == BFS_ALLOC_PER_INSTR) {
    for (auto &kv : slot_of_instr) p.instr_update[kv.first] = kv.second;
    p.n_counters = (int32_t)slot_of_instr.size();
  } else if (p.alloc == BFS_ALLOC_PER_ENGINE) {
    for (int32_t i = 0; i < I; ++i) {
      auto it = slot_of_engine.find(p.instr_engine[i]);
      if (it != slot_of_engine.end()) p.instr_update[i] = it->second;
    }
    p.n_counters = (int32_t)slot_of_engine.size();
  } else {
    for (int32_t i = 0; i < I; ++i) {
      auto it = slot_of_loop_engine.find({p.instr_parent[i], p.instr_engine[i]});
      if (it != slot_of_loop_engine.end()) p.instr_update[i] = it->second;
    }
    p.n_counters = (int32_t)slot_of_loop_engine.size();
  }
  if (p.n_counters > kMaxSlots) return fail(BFS_E_RESOURCE, "more than 64 counter slots");

  // Per-instruction wait lists.
  p.instr_wait_off.assign(I + 1, 0);
  p.instr_wait_list.clear();
  for (int32_t i = 0; i < I; ++i) {
    p.instr_wait_off[i] = (int32_t)p.instr_wait_list.size();
    for (int32_t d = 0; d < D; ++d)
      if (p.deps[3 * d + 1] == i) {
        bool needed = p.mode == BFS_MODE_BARRIER_FREE ? p.formulas[d].kase != 4 : p.static_waits[d].same_region != 0;
        if (needed) p.instr_wait_list.push_back(d);
      }
  }
  p.instr_wait_off[I] = (int32_t)p.instr_wait_list.size();

  // Per-engine allocation: each consumer engine's snapshot area holds one
  // running count per engine (words 0 .. kMaxEngines - 1), then the
  // snapshots of its dependencies in dependency order.
  p.snap_off.assign(D, 0);
  p.snap_words = 0;
  const bool per_engine = p.mode == BFS_MODE_BARRIER_FREE && p.alloc == BFS_ALLOC_PER_ENGINE;
  std::vector<std::vector<char>> tracks(E, std::vector<char>(kMaxEngines, 0));   // consumer -> producer engines
  if (per_engine) {
    std::vector<int32_t> used(E, kMaxEngines);
    for (int32_t d = 0; d < D; ++d) {
      const bfs_formula &f = p.formulas[d];
      if (f.kase == 4) continue;
      p.snap_off[d] = used[f.cns_engine];
      used[f.cns_engine] += f.snap_slots;
      tracks[f.cns_engine][f.prd_engine] = 1;
    }
    for (int32_t e = 0; e < E; ++e) p.snap_words = std::max(p.snap_words, used[e]);
  }

  // Interpreter code: each engine's projection of the statement tree.
  p.code.clear();
  p.code_off.assign(E + 1, 0);
  for (int32_t e = 0; e < E; ++e) {
    p.code_off[e] = (int32_t)p.code.size() / 4;
    std::vector<int32_t> &C = p.code;
    const int32_t base = p.code_off[e];
    auto emit = [&](int32_t kind, int32_t a0, int32_t a1) {
      C.push_back(kind); C.push_back(a0); C.push_back(a1); C.push_back(0);
      return (int32_t)C.size() / 4 - 1 - base;
    };
    // iterative depth-first emission
    struct Frame { int32_t loop, it, pc; };
    std::vector<Frame> fr{{0, p.body_off[0], -1}};
    while (!fr.empty()) {
      Frame &f = fr.back();
      if (f.it == p.body_off[f.loop + 1]) {
        if (f.loop != 0) {
          int32_t endpc = emit(CODE_END, f.loop, f.pc);
          C[4 * (base + f.pc) + 2] = endpc;      // loop word points at its end word
        }
        fr.pop_back();
        continue;
      }
      int32_t kind = p.body_kind[f.it], id = p.body_id[f.it];
      ++f.it;
      if (kind == 0) {
        // Per-engine: the counts of the tracked producer engines' instructions
        // are added as the block is passed (once per execution of the block),
        // flushed before every snapshot and at the block's end.
        int32_t pend[kMaxEngines] = {0};
        auto flush = [&](int32_t pe) {
          if (pend[pe] > 0) emit(CODE_TRACK, pe, pend[pe]);
          pend[pe] = 0;
        };
        for (int32_t j = p.block_off[id]; j < p.block_off[id + 1]; ++j) {
          const int32_t ins = p.block_instrs[j], ie = p.instr_engine[ins];
          if (ie == e) emit(CODE_INSTR, ins, 0);
          if (!per_engine || !tracks[e][ie]) continue;
          pend[ie] += 1;
          for (int32_t d = 0; d < D; ++d)
            if (p.deps[3 * d] == ins && p.formulas[d].kase != 4 && p.formulas[d].cns_engine == e) {
              flush(ie);
              emit(CODE_SNAP, d, 0);
            }
        }
        for (int32_t pe = 0; pe < E; ++pe) flush(pe);
      } else {
        int32_t pc = emit(CODE_LOOP, id, -1);
        fr.push_back(Frame{id, p.body_off[id], pc});
      }
    }
    emit(CODE_HALT, 0, 0);
  }
  p.code_off[E] = (int32_t)p.code.size() / 4;

  // Resource figures.
  bfs_stats s{};
  s.n_counters = p.n_counters;
  int32_t syncs = 0;
  for (int32_t l = 1; l < L; ++l) syncs += 2;
  s.n_sync_points = syncs;
  if (p.mode == BFS_MODE_BARRIER) {
    s.regs_per_engine = 0;
    s.salu_ops_per_wait = 0;
    for (auto &w : p.static_waits) s.n_waits += w.same_region;
  } else {
    std::vector<char> usedP(L, 0), usedS(L, 0);
    for (auto &f : p.formulas) {
      if (f.kase == 4) continue;
      usedP[f.loop_P] = 1;
      if (f.needs_mask) usedS[f.loop_S] = 1;
    }
    int32_t regs = 1;   // the wait register
    for (int32_t l = 0; l < L; ++l) regs += usedP[l] + usedS[l];
    if (per_engine) {
      // running counts of the tracked engines and the snapshots, most of any engine
      int32_t extra = 0;
      for (int32_t e = 0; e < E; ++e) {
        int32_t x = 0;
        for (int32_t pe = 0; pe < kMaxEngines; ++pe) x += tracks[e][pe];
        for (int32_t d = 0; d < D; ++d)
          if (p.formulas[d].kase != 4 && p.formulas[d].cns_engine == e) x += p.formulas[d].snap_slots;
        extra = std::max(extra, x);
      }
      regs += extra;
    }
    s.regs_per_engine = regs;
    s.salu_ops_per_wait = p.alloc == BFS_ALLOC_PER_INSTR ? 3 : p.alloc == BFS_ALLOC_PER_ENGINE ? 3 : 5;
    s.n_sync_points = __builtin_popcount(p.fallback_loops);
    s.n_waits = 0;
    for (auto &f : p.formulas) s.n_waits += f.kase != 4;
  }
  for (auto &f : p.formulas) s.n_fallback += f.kase == 4;
  p.stats = s;
  return BFS_OK;
}

uint32_t eval_formula(const bfs_formula &f, uint32_t r_P, uint32_t rhat_S) {
  if (f.needs_mask && !(rhat_S > (uint32_t)f.k)) return 0;
  int64_t v = (int64_t)f.N * ((int64_t)r_P - f.expr_sub) - (f.N - f.K);
  return v > 0 ? (uint32_t)v : 0u;
}

}  // namespace bfs

using namespace bfs;

extern "C" {

bfs_status bfs_plan_create(const bfs_program *prog, bfs_mode mode, bfs_alloc alloc, uint32_t flags,
                           bfs_plan **out) {
  if (!prog || !out) return fail(BFS_E_INVALID, "null argument");
  if (flags & ~BFS_PLAN_BARRIER_FALLBACK) return fail(BFS_E_INVALID, "unknown plan flags");
  if (mode != BFS_MODE_BARRIER_FREE && mode != BFS_MODE_BARRIER) return fail(BFS_E_INVALID, "bad mode");
  if (alloc != BFS_ALLOC_PER_LOOP && alloc != BFS_ALLOC_PER_INSTR && alloc != BFS_ALLOC_PER_ENGINE)
    return fail(BFS_E_INVALID, "bad alloc");
  if (prog->kernel < BFS_KERNEL_INTERP || prog->kernel > BFS_KERNEL_CHAIN) return fail(BFS_E_INVALID, "bad kernel");
  if (prog->n_loops < 1 || prog->n_blocks < 0 || prog->n_instrs < 0 || prog->n_deps < 0)
    return fail(BFS_E_INVALID, "negative sizes");
  if (!prog->loop_parent || !prog->body_off || !prog->block_off)
    return fail(BFS_E_INVALID, "null program array");
  bfs_plan *p = new bfs_plan();
  static std::atomic<uint64_t> next_uid{1};
  p->uid = next_uid.fetch_add(1);
  p->mode = mode;
  p->alloc = alloc;
  p->kernel = prog->kernel;
  p->n_engines = prog->n_engines;
  for (int e = 0; e < kMaxEngines; ++e) p->waves_per_engine[e] = prog->waves_per_engine[e];
  p->n_loops = prog->n_loops;
  const int32_t L = prog->n_loops, B = prog->n_blocks, I = prog->n_instrs, D = prog->n_deps;
  p->loop_parent.assign(prog->loop_parent, prog->loop_parent + L);
  p->loop_is_cond.assign(L, 0);
  if (prog->loop_is_cond) p->loop_is_cond.assign(prog->loop_is_cond, prog->loop_is_cond + L);
  p->body_off.assign(prog->body_off, prog->body_off + L + 1);
  int32_t nb = p->body_off[L];
  if (nb < 0 || (nb > 0 && (!prog->body_kind || !prog->body_id))) {
    delete p;
    return fail(BFS_E_INVALID, "bad body arrays");
  }
  p->body_kind.assign(prog->body_kind, prog->body_kind + nb);
  p->body_id.assign(prog->body_id, prog->body_id + nb);
  p->block_off.assign(prog->block_off, prog->block_off + B + 1);
  int32_t ni = p->block_off[B];
  if (ni != I || (I > 0 && (!prog->block_instrs || !prog->instr_engine || !prog->instr_opcode || !prog->instr_args))) {
    delete p;
    return fail(BFS_E_INVALID, "blocks must list every instruction once");
  }
  p->block_instrs.assign(prog->block_instrs, prog->block_instrs + I);
  p->instr_engine.assign(prog->instr_engine, prog->instr_engine + I);
  p->instr_opcode.assign(prog->instr_opcode, prog->instr_opcode + I);
  p->instr_args.assign(prog->instr_args, prog->instr_args + 8 * (size_t)I);
  if (D > 0 && !prog->deps) {
    delete p;
    return fail(BFS_E_INVALID, "null deps");
  }
  p->deps.assign(prog->deps, prog->deps + 3 * (size_t)D);
  p->dep_linear.assign(D, 0);
  if (prog->dep_linear) p->dep_linear.assign(prog->dep_linear, prog->dep_linear + D);
  p->tile_elems = prog->tile_elems;
  for (int r = 0; r < 4; ++r) p->ring_slots[r] = prog->ring_slots[r];
  p->n_accs = prog->n_accs;
  p->flags = flags;
  bfs_status st = plan_build(*p);
  if (st != BFS_OK) {
    delete p;
    return st;
  }
  *out = p;
  return BFS_OK;
}

bfs_status bfs_plan_formulas(const bfs_plan *plan, const bfs_formula **out, int32_t *n) {
  if (!plan || !out || !n) return fail(BFS_E_INVALID, "null argument");
  *out = plan->formulas.data();
  *n = (int32_t)plan->formulas.size();
  return BFS_OK;
}

bfs_status bfs_plan_static_waits(const bfs_plan *plan, const bfs_static_wait **out, int32_t *n) {
  if (!plan || !out || !n) return fail(BFS_E_INVALID, "null argument");
  *out = plan->static_waits.data();
  *n = (int32_t)plan->static_waits.size();
  return BFS_OK;
}

bfs_status bfs_plan_stats(const bfs_plan *plan, bfs_stats *out) {
  if (!plan || !out) return fail(BFS_E_INVALID, "null argument");
  *out = plan->stats;
  return BFS_OK;
}

bfs_status bfs_eval_threshold(const bfs_plan *plan, int32_t dep, uint32_t r_P, uint32_t rhat_S, uint32_t *out) {
  if (!plan || !out) return fail(BFS_E_INVALID, "null argument");
  if (dep < 0 || dep >= (int32_t)plan->formulas.size()) return fail(BFS_E_INVALID, "bad dependency id");
  if (plan->mode == BFS_MODE_BARRIER) {
    const bfs_static_wait &w = plan->static_waits[dep];
    *out = w.same_region ? (uint32_t)w.ordinal : 0u;
  } else if (plan->formulas[dep].kase == 4) {
    *out = 0u;
  } else if (plan->alloc == BFS_ALLOC_PER_ENGINE) {
    return fail(BFS_E_UNSUPPORTED, "per-engine thresholds are snapshots taken during the walk, not a function "
                                   "of r_P and rhat_S");
  } else {
    *out = eval_formula(plan->formulas[dep], r_P, rhat_S);
  }
  return BFS_OK;
}

void bfs_plan_destroy(bfs_plan *plan) {
  if (!plan) return;
  free_images(plan);
  delete plan;
}

const char *bfs_status_string(bfs_status s) {
  switch (s) {
    case BFS_OK: return "ok";
    case BFS_E_INVALID: return "invalid argument or program";
    case BFS_E_ORDER: return "producer does not precede consumer";
    case BFS_E_NOT_ALLOCATABLE: return "dependency not allocatable";
    case BFS_E_RESOURCE: return "resource limit exceeded";
    case BFS_E_DEVICE: return "device error";
    case BFS_E_DEADLOCK: return "device wait exceeded the watchdog";
    case BFS_E_UNSUPPORTED: return "unsupported by the kernel family";
  }
  return "unknown status";
}

const char *bfs_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
