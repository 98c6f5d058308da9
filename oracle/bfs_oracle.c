/*
 * CPU oracle for barrier-free multi-engine synchronization.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this file.  It shares no code with the GPU
 * library: it reads the same program description and the same seeded inputs
 * and recomputes everything from the definitions in the paper.
 *
 * What it computes, for one workgroup:
 *
 *  1. A sequential program-order execution of the structured program
 *     (Section 4.1: every construct is a loop; the program is a top-level
 *     loop that runs once).  Each executed instruction instance is recorded
 *     with the iteration number of every enclosing loop in its current trip
 *     (the iteration vector of Section 4.1, 1-based) and the total number of
 *     entries of every loop so far.  The tile-machine datapath semantics are
 *     applied in fp64, giving the reference values: any schedule that
 *     respects the dependencies produces the same values.
 *
 *  2. For every dependency (p, c, k) and every executed instance of c: the
 *     producer-completion count demanded by the dependency-satisfaction
 *     condition, Eq. (1) of Section 4.2, by brute force.  With S the innermost
 *     loop enclosing both p and c, the target t is the consumer's iteration
 *     vector over the loops from the top level down to S with the S component
 *     reduced by k.  If that component is <= 0 the target underflows and
 *     nothing is owed; otherwise the count is the number of executed
 *     instances of p whose iteration vector over the same loops is
 *     lexicographically <= t.
 *
 *  3. The same requirement expressed on the per-loop semaphore of Section 5.5:
 *     one counter per (loop, engine), incremented at the retirement of every
 *     instruction of that engine whose innermost enclosing loop is that loop.
 *     The semaphore threshold is the counter value right after the latest
 *     retirement among the counted producer instances (0 if none).
 *
 *  5. The same requirement expressed on the per-engine semaphore of
 *     Section 6.1: one counter per engine, incremented at the retirement of
 *     every instruction of that engine (in-order retirement makes its value
 *     the number of the engine's instructions retired so far).  The threshold
 *     is that counter's value right after the latest counted producer
 *     instance (0 if none).
 *
 *  4. The barrier-based scheme of Section 3.4: all engines synchronize before
 *     every non-top loop statement and at the end of every iteration of a
 *     non-top loop, resetting one counter per engine.  A consumer instance
 *     whose latest required producer instance lies in the same barrier region
 *     waits for that producer's ordinal on its engine since the last barrier;
 *     otherwise the barrier already ordered it and the threshold is 0.
 *
 * Everything is counted by simulation; no closed form is used.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_MAX_LOOPS 64
#define ORC_MAX_ENGINES 8

/* Tile-machine opcodes, as documented with the program description. */
enum { ORC_NOP = 0, ORC_LOAD = 1, ORC_SCALE_ACC = 2, ORC_STORE_ACC = 3, ORC_ADDC = 4, ORC_STORE_RING = 5 };

typedef struct {
  int32_t n_engines, n_loops, n_blocks, n_instrs, n_deps;
  const int32_t *loop_parent;               /* [n_loops], top = -1 */
  const int32_t *body_off;                  /* [n_loops + 1] */
  const int32_t *body_kind, *body_id;       /* [body_off[n_loops]] ; 0 block, 1 loop */
  const int32_t *block_off;                 /* [n_blocks + 1] */
  const int32_t *block_instrs;              /* [block_off[n_blocks]] */
  const int32_t *instr_engine, *instr_opcode;
  const int32_t *instr_args;                /* [n_instrs][8] */
  const int32_t *deps;                      /* [n_deps][3] = producer, consumer, offset */
  int32_t tile_elems, n_rings, n_accs;
  const int32_t *ring_slots;                /* [n_rings] */
} orc_prog;

/* One executed instruction instance. */
typedef struct {
  int32_t instr, engine;
  int64_t cnt_after;      /* per-loop counter (parent loop, engine) after its retirement */
  int64_t cnt_before;     /* value of that counter just before it issued */
  int64_t region;         /* barrier region id */
  int64_t bord;           /* ordinal on its engine within the barrier region */
  int64_t ecnt_after;     /* per-engine counter (every instruction of the engine) after its retirement */
} orc_inst;

/* One consumer instance of one dependency. */
typedef struct {
  int32_t dep;
  int32_t instance;       /* 0-based execution index of the consumer */
  int64_t count_thr;      /* producer completions owed (Eq. 1) */
  int64_t sem_thr;        /* per-loop counter value that certifies them */
  int64_t barrier_thr;    /* barrier-based scheme's static threshold */
  int64_t r_P, r_S, rhat_S; /* entry counts at the consumer's issue */
  int32_t order_ok;       /* program order already satisfies the requirement */
  int32_t pad;
  int64_t eng_thr;        /* per-engine counter value that certifies them */
} orc_rec;

typedef struct {
  const orc_prog *P;
  const int32_t *trips;
  const int64_t *trip_off;      /* [n_loops] for this workgroup */
  int64_t exec_count[ORC_MAX_LOOPS];
  int64_t r[ORC_MAX_LOOPS];     /* entries of each loop since the start */
  int64_t rhat[ORC_MAX_LOOPS];  /* entries in the current trip */
  int64_t *cnt;                 /* [n_loops * n_engines] per-loop counters */
  int64_t bcnt[ORC_MAX_ENGINES];
  int64_t ecnt[ORC_MAX_ENGINES];  /* per-engine counters */
  int64_t region;
  int64_t n_inst;
  int64_t cap;
  orc_inst *inst;               /* may be NULL (counting pass) */
  int32_t *r_snap, *rhat_snap;  /* [cap][n_loops] */
  /* datapath state, fp64 */
  int64_t wg;
  const int64_t *base;
  const float *x;
  double *out;
  int64_t out_len;
  double *rings[4];
  double *accs;
  int err;
} orc_state;

static int parent_of_instr(const orc_prog *P, int32_t instr, int32_t *owner_loop) {
  /* The innermost loop whose body lists the block holding instr. */
  for (int32_t l = 0; l < P->n_loops; ++l)
    for (int32_t it = P->body_off[l]; it < P->body_off[l + 1]; ++it)
      if (P->body_kind[it] == 0) {
        int32_t b = P->body_id[it];
        for (int32_t j = P->block_off[b]; j < P->block_off[b + 1]; ++j)
          if (P->block_instrs[j] == instr) { *owner_loop = l; return 0; }
      }
  return -1;
}

static int64_t slot_of(const orc_state *st, const int32_t *a) {
  /* slot = ((r[gen]-1) % n_gen) * per_gen + ((rhat[pos]-1) % per_gen) */
  int64_t hi = 0;
  if (a[2] >= 0) hi = ((st->r[a[2]] - 1) % a[3]) * a[5];
  int64_t lo = (a[4] >= 0) ? ((st->rhat[a[4]] - 1) % a[5]) : 0;
  return hi + lo;
}

static void datapath(orc_state *st, int32_t instr) {
  const orc_prog *P = st->P;
  const int32_t *a = P->instr_args + 8 * instr;
  int32_t T = P->tile_elems;
  float cf;
  memcpy(&cf, &a[7], 4);
  double c = (double)cf;
  switch (P->instr_opcode[instr]) {
    case ORC_NOP: break;
    case ORC_LOAD: {
      int64_t g = st->base[st->wg] + st->r[a[6]] - 1;
      double *dst = st->rings[a[1]] + slot_of(st, a) * T;
      for (int32_t e = 0; e < T; ++e) dst[e] = (double)st->x[g * T + e];
      break;
    }
    case ORC_SCALE_ACC: {
      const double *src = st->rings[a[0]] + slot_of(st, a) * T;
      double *acc = st->accs + (int64_t)a[1] * T;
      for (int32_t e = 0; e < T; ++e) acc[e] += c * src[e];
      break;
    }
    case ORC_STORE_ACC: {
      const double *acc = st->accs + (int64_t)a[0] * T;
      for (int32_t e = 0; e < T; ++e) st->out[st->wg * T + e] = acc[e];
      break;
    }
    case ORC_ADDC: {
      int64_t s = slot_of(st, a);
      const double *src = st->rings[a[0]] + s * T;
      double *dst = st->rings[a[1]] + s * T;
      for (int32_t e = 0; e < T; ++e) dst[e] = src[e] + c;
      break;
    }
    case ORC_STORE_RING: {
      int64_t g = st->base[st->wg] + st->r[a[6]] - 1;
      const double *src = st->rings[a[0]] + slot_of(st, a) * T;
      for (int32_t e = 0; e < T; ++e) st->out[g * T + e] = src[e];
      break;
    }
    default: break;   /* descriptive opcodes carry no tile-machine effect */
  }
}

static void exec_instr(orc_state *st, int32_t instr, int32_t parent) {
  const orc_prog *P = st->P;
  int32_t e = P->instr_engine[instr];
  int64_t *c = &st->cnt[(int64_t)parent * P->n_engines + e];
  int64_t idx = st->n_inst++;
  if (st->inst) {
    if (idx >= st->cap) { st->err = 1; return; }
    orc_inst *I = &st->inst[idx];
    I->instr = instr;
    I->engine = e;
    I->cnt_before = *c;
    I->region = st->region;
    for (int32_t l = 0; l < P->n_loops; ++l) {
      st->r_snap[idx * P->n_loops + l] = (int32_t)st->r[l];
      st->rhat_snap[idx * P->n_loops + l] = (int32_t)st->rhat[l];
    }
    if (st->x || st->out) datapath(st, instr);
  }
  *c += 1;
  st->bcnt[e] += 1;
  st->ecnt[e] += 1;
  if (st->inst) {
    st->inst[idx].cnt_after = *c;
    st->inst[idx].bord = st->bcnt[e];
    st->inst[idx].ecnt_after = st->ecnt[e];
  }
}

static void barrier_sync(orc_state *st) {
  st->region += 1;
  for (int e = 0; e < ORC_MAX_ENGINES; ++e) st->bcnt[e] = 0;
}

static void walk_body(orc_state *st, int32_t l) {
  const orc_prog *P = st->P;
  for (int32_t it = P->body_off[l]; it < P->body_off[l + 1] && !st->err; ++it) {
    int32_t id = P->body_id[it];
    if (P->body_kind[it] == 0) {
      for (int32_t j = P->block_off[id]; j < P->block_off[id + 1]; ++j)
        exec_instr(st, P->block_instrs[j], l);
    } else {
      int64_t trip = st->trips[st->trip_off[id] + st->exec_count[id]];
      st->exec_count[id] += 1;
      barrier_sync(st);                 /* before the loop statement */
      st->rhat[id] = 0;
      for (int64_t i = 0; i < trip && !st->err; ++i) {
        st->r[id] += 1;
        st->rhat[id] += 1;
        walk_body(st, id);
        barrier_sync(st);               /* end of the iteration */
      }
    }
  }
}

static void run_walk(orc_state *st) {
  memset(st->exec_count, 0, sizeof st->exec_count);
  memset(st->r, 0, sizeof st->r);
  memset(st->rhat, 0, sizeof st->rhat);
  memset(st->bcnt, 0, sizeof st->bcnt);
  memset(st->ecnt, 0, sizeof st->ecnt);
  st->region = 0;
  st->n_inst = 0;
  st->r[0] = 1;                          /* the program is a loop entered once */
  st->rhat[0] = 1;
  walk_body(st, 0);
}

/* Number of instruction instances executed by one workgroup. */
int64_t orc_count_instances(const orc_prog *P, const int32_t *trips, const int64_t *trip_off) {
  if (P->n_loops > ORC_MAX_LOOPS || P->n_engines > ORC_MAX_ENGINES) return -1;
  orc_state st;
  memset(&st, 0, sizeof st);
  st.P = P;
  st.trips = trips;
  st.trip_off = trip_off;
  st.cnt = (int64_t *)calloc((size_t)P->n_loops * P->n_engines, sizeof(int64_t));
  run_walk(&st);
  free(st.cnt);
  return st.n_inst;
}

/* Loops from the top level down to l (inclusive); returns the depth. */
static int32_t path_to(const orc_prog *P, int32_t l, int32_t *path) {
  int32_t tmp[ORC_MAX_LOOPS], n = 0;
  for (int32_t x = l; x >= 0; x = P->loop_parent[x]) tmp[n++] = x;
  for (int32_t i = 0; i < n; ++i) path[i] = tmp[n - 1 - i];
  return n;
}

static int32_t innermost_common(const orc_prog *P, int32_t a, int32_t b) {
  int32_t pa[ORC_MAX_LOOPS], pb[ORC_MAX_LOOPS];
  int32_t na = path_to(P, a, pa), nb = path_to(P, b, pb);
  int32_t s = 0;
  for (int32_t i = 0; i < na && i < nb && pa[i] == pb[i]; ++i) s = pa[i];
  return s;
}

/*
 * Full oracle pass for one workgroup.
 *   inst/r_snap/rhat_snap: trace buffers sized by orc_count_instances().
 *   recs: one record per (dependency, consumer instance), rec_cap entries.
 *   final_cnt: [n_loops][n_engines] per-loop counters at the end.
 *   base/x/out may be NULL when only thresholds are wanted.
 * Returns 0 on success, negative on error.
 */
int orc_run(const orc_prog *P, const int32_t *trips, const int64_t *trip_off, int64_t wg,
            const int64_t *base, const float *x, double *out, int64_t out_len,
            orc_inst *inst, int32_t *r_snap, int32_t *rhat_snap, int64_t cap,
            orc_rec *recs, int64_t rec_cap, int64_t *n_recs, int64_t *final_cnt) {
  if (P->n_loops > ORC_MAX_LOOPS || P->n_engines > ORC_MAX_ENGINES) return -1;
  orc_state st;
  memset(&st, 0, sizeof st);
  st.P = P;
  st.trips = trips;
  st.trip_off = trip_off;
  st.cap = cap;
  st.inst = inst;
  st.r_snap = r_snap;
  st.rhat_snap = rhat_snap;
  st.wg = wg;
  st.base = base;
  st.x = x;
  st.out = out;
  st.out_len = out_len;
  st.cnt = (int64_t *)calloc((size_t)P->n_loops * P->n_engines, sizeof(int64_t));
  int64_t T = P->tile_elems > 0 ? P->tile_elems : 1;
  for (int32_t i = 0; i < P->n_rings && i < 4; ++i)
    st.rings[i] = (double *)calloc((size_t)(P->ring_slots[i] > 0 ? P->ring_slots[i] : 1) * T, sizeof(double));
  st.accs = (double *)calloc((size_t)(P->n_accs > 0 ? P->n_accs : 1) * T, sizeof(double));
  run_walk(&st);
  int rc = st.err ? -2 : 0;
  if (final_cnt) memcpy(final_cnt, st.cnt, sizeof(int64_t) * (size_t)P->n_loops * P->n_engines);

  /* Thresholds by brute force over the recorded trace. */
  int64_t nr = 0;
  int32_t *parent = (int32_t *)malloc(sizeof(int32_t) * (size_t)(P->n_instrs > 0 ? P->n_instrs : 1));
  for (int32_t i = 0; i < P->n_instrs; ++i)
    if (parent_of_instr(P, i, &parent[i]) != 0) rc = -3;
  int64_t L = P->n_loops;
  for (int32_t d = 0; d < P->n_deps && rc == 0; ++d) {
    int32_t p = P->deps[3 * d], c = P->deps[3 * d + 1], k = P->deps[3 * d + 2];
    int32_t S = innermost_common(P, parent[p], parent[c]);
    int32_t path[ORC_MAX_LOOPS];
    int32_t depth = path_to(P, S, path);
    int32_t instance = 0;
    for (int64_t xi = 0; xi < st.n_inst; ++xi) {
      if (inst[xi].instr != c) continue;
      int64_t t[ORC_MAX_LOOPS];
      for (int32_t j = 0; j < depth; ++j) t[j] = rhat_snap[xi * L + path[j]];
      t[depth - 1] -= k;
      int64_t count = 0, sem = 0, bthr = 0, eng = 0;
      int64_t latest = -1;
      if (t[depth - 1] > 0) {
        for (int64_t yi = 0; yi < st.n_inst; ++yi) {
          if (inst[yi].instr != p) continue;
          int le = 1;      /* lexicographic <= over the loops top..S */
          for (int32_t j = 0; j < depth; ++j) {
            int64_t v = rhat_snap[yi * L + path[j]];
            if (v < t[j]) { le = 1; break; }
            if (v > t[j]) { le = 0; break; }
          }
          if (!le) continue;
          count += 1;
          if (inst[yi].cnt_after > sem) { sem = inst[yi].cnt_after; latest = yi; }
          if (inst[yi].ecnt_after > eng) eng = inst[yi].ecnt_after;
        }
      }
      if (latest >= 0 && inst[latest].region == inst[xi].region) bthr = inst[latest].bord;
      if (nr < rec_cap) {
        orc_rec *R = &recs[nr];
        R->dep = d;
        R->instance = instance;
        R->count_thr = count;
        R->sem_thr = sem;
        R->eng_thr = eng;
        R->barrier_thr = bthr;
        R->r_P = r_snap[xi * L + parent[p]];
        R->r_S = r_snap[xi * L + S];
        R->rhat_S = rhat_snap[xi * L + S];
        /* counter (parent(p), engine(p)) at the consumer's program-order position */
        int64_t at = 0;
        for (int64_t yi = xi - 1; yi >= 0; --yi)
          if (inst[yi].engine == P->instr_engine[p] && parent[inst[yi].instr] == parent[p]) {
            at = inst[yi].cnt_after;
            break;
          }
        R->order_ok = at >= sem;
      }
      nr += 1;
      instance += 1;
    }
  }
  *n_recs = nr;
  free(parent);
  for (int i = 0; i < 4; ++i) free(st.rings[i]);
  free(st.accs);
  free(st.cnt);
  return rc;
}

/* Sequential walk that rewinds a one-entry trace after every instance. */
static void walk_values(orc_state *st, int32_t l) {
  const orc_prog *P = st->P;
  for (int32_t it = P->body_off[l]; it < P->body_off[l + 1] && !st->err; ++it) {
    int32_t id = P->body_id[it];
    if (P->body_kind[it] == 0) {
      for (int32_t j = P->block_off[id]; j < P->block_off[id + 1]; ++j) {
        st->n_inst = 0;
        exec_instr(st, P->block_instrs[j], l);
      }
    } else {
      int64_t trip = st->trips[st->trip_off[id] + st->exec_count[id]];
      st->exec_count[id] += 1;
      st->rhat[id] = 0;
      for (int64_t i = 0; i < trip && !st->err; ++i) {
        st->r[id] += 1;
        st->rhat[id] += 1;
        walk_values(st, id);
      }
    }
  }
}

/*
 * Values only, for many workgroups (the reference result of a tile-machine
 * workload).  Runs the same sequential walk without recording thresholds.
 */
int orc_values(const orc_prog *P, const int32_t *trips, const int64_t *trip_off_all, int64_t n_wg,
               const int64_t *base, const float *x, double *out, int64_t out_len) {
  if (P->n_loops > ORC_MAX_LOOPS || P->n_engines > ORC_MAX_ENGINES) return -1;
  int64_t T = P->tile_elems > 0 ? P->tile_elems : 1;
  orc_state st;
  memset(&st, 0, sizeof st);
  st.P = P;
  st.trips = trips;
  st.base = base;
  st.x = x;
  st.out = out;
  st.out_len = out_len;
  st.cnt = (int64_t *)calloc((size_t)P->n_loops * P->n_engines, sizeof(int64_t));
  for (int32_t i = 0; i < P->n_rings && i < 4; ++i)
    st.rings[i] = (double *)calloc((size_t)(P->ring_slots[i] > 0 ? P->ring_slots[i] : 1) * T, sizeof(double));
  st.accs = (double *)calloc((size_t)(P->n_accs > 0 ? P->n_accs : 1) * T, sizeof(double));
  /* one-instance scratch trace: datapath() only needs the live registers */
  orc_inst one;
  int32_t *rs = (int32_t *)calloc((size_t)P->n_loops, sizeof(int32_t));
  int32_t *rh = (int32_t *)calloc((size_t)P->n_loops, sizeof(int32_t));
  for (int64_t w = 0; w < n_wg; ++w) {
    st.wg = w;
    st.trip_off = trip_off_all + w * P->n_loops;
    memset(st.cnt, 0, sizeof(int64_t) * (size_t)P->n_loops * P->n_engines);
    for (int32_t a = 0; a < P->n_accs; ++a)
      memset(st.accs + a * T, 0, sizeof(double) * (size_t)T);
    /* run with a trace of capacity 1 that is rewound after each instance */
    st.inst = &one;
    st.r_snap = rs;
    st.rhat_snap = rh;
    st.cap = 1;
    memset(st.exec_count, 0, sizeof st.exec_count);
    memset(st.r, 0, sizeof st.r);
    memset(st.rhat, 0, sizeof st.rhat);
    st.r[0] = 1;
    st.rhat[0] = 1;
    st.n_inst = 0;
    st.err = 0;
    walk_values(&st, 0);
    if (st.err) break;
  }
  int rc = st.err ? -2 : 0;
  free(rs);
  free(rh);
  for (int i = 0; i < 4; ++i) free(st.rings[i]);
  free(st.accs);
  free(st.cnt);
  return rc;
}
