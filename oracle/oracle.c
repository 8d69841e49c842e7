/*
 * oracle.c -- plain CPU reference scorer (TEST INFRASTRUCTURE ONLY; see
 * oracle.h).  Written for readability, not speed: one plan at a time, the
 * steps in the order the paper's scheduler applies them, int64 arithmetic
 * for every time and memory sum, no blocking, no fusion of steps.
 *
 * Build: gcc -O2 -std=c99 -ffp-contract=off -fPIC -shared (no fused
 * multiply-add: the objective is two fp32 products and one fp32 sum, each
 * rounded to nearest even).
 */
#include "oracle.h"

#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------------- */
/* window structure                                                        */
/* ---------------------------------------------------------------------- */

typedef struct {
  int32_t *level;    /* topological level                                */
  int32_t *n_succ;   /* number of successors                             */
  int32_t *child;    /* the successor when n_succ == 1, else -1          */
  uint8_t *fusible;  /* Eq. 3: single pred u, u has single succ, same model */
} orc_struct;

static void free_struct(orc_struct *s) {
  free(s->level);
  free(s->n_succ);
  free(s->child);
  free(s->fusible);
}

static int build_struct(const orc_window *w, orc_struct *s) {
  const int32_t N = w->n_act;
  memset(s, 0, sizeof *s);
  if (N < 0 || w->n_wf < 0 || w->n_models < 1 || w->n_models > 64 || w->n_dev < 1)
    return ORC_ERR_SIZE;
  if (N > 0 && w->n_wf < 1) return ORC_ERR_SIZE;
  size_t n = (size_t)(N > 0 ? N : 1);
  s->level = (int32_t *)calloc(n, sizeof(int32_t));
  s->n_succ = (int32_t *)calloc(n, sizeof(int32_t));
  s->child = (int32_t *)calloc(n, sizeof(int32_t));
  s->fusible = (uint8_t *)calloc(n, 1);
  if (!s->level || !s->n_succ || !s->child || !s->fusible) {
    free_struct(s);
    return ORC_ERR_NOMEM;
  }
  /* levels: a source is level 0, otherwise one more than its deepest pred */
  for (int32_t i = 0; i < N; ++i) {
    int32_t lv = 0;
    for (int32_t k = w->pred_off[i]; k < w->pred_off[i + 1]; ++k) {
      int32_t p = w->pred_idx[k];
      if (p < 0 || p >= i) return free_struct(s), ORC_ERR_PRED;
      if (k > w->pred_off[i] && p <= w->pred_idx[k - 1]) return free_struct(s), ORC_ERR_PRED;
      if (s->level[p] + 1 > lv) lv = s->level[p] + 1;
    }
    s->level[i] = lv;
    if (i > 0 && lv < s->level[i - 1]) return free_struct(s), ORC_ERR_ORDER;
    if (w->act_wf[i] < 0 || w->act_wf[i] >= w->n_wf) return free_struct(s), ORC_ERR_INDEX;
    if (w->act_model[i] < 0 || w->act_model[i] >= w->n_models)
      return free_struct(s), ORC_ERR_INDEX;
  }
  /* every workflow has at least one activation */
  for (int32_t wf = 0; wf < w->n_wf; ++wf) {
    int found = 0;
    for (int32_t i = 0; i < N && !found; ++i) found = (w->act_wf[i] == wf);
    if (!found) return free_struct(s), ORC_ERR_EMPTY_WF;
  }
  /* successor counts and the unique successor */
  for (int32_t i = 0; i < N; ++i) s->child[i] = -1;
  for (int32_t v = 0; v < N; ++v)
    for (int32_t k = w->pred_off[v]; k < w->pred_off[v + 1]; ++k) {
      int32_t u = w->pred_idx[k];
      s->n_succ[u] += 1;
      s->child[u] = v;
    }
  for (int32_t u = 0; u < N; ++u)
    if (s->n_succ[u] != 1) s->child[u] = -1;
  /* Eq. 3: edge (u, v) is fusible when pred(v) = {u}, succ(u) = {v} and both
   * need the same deployment (every node is an agent node; one serving
   * configuration per model) */
  for (int32_t v = 0; v < N; ++v) {
    if (w->pred_off[v + 1] - w->pred_off[v] != 1) continue;
    int32_t u = w->pred_idx[w->pred_off[v]];
    s->fusible[v] = (s->n_succ[u] == 1 && w->act_model[u] == w->act_model[v]);
  }
  return ORC_OK;
}

int orc_levels(const orc_window *w, int32_t *level_out) {
  orc_struct s;
  int rc = build_struct(w, &s);
  if (rc) return rc;
  for (int32_t i = 0; i < w->n_act; ++i) level_out[i] = s.level[i];
  free_struct(&s);
  return ORC_OK;
}

/* ---------------------------------------------------------------------- */
/* ordering                                                                */
/* ---------------------------------------------------------------------- */

typedef struct {
  int32_t level;
  int32_t prio;
  int32_t idx;
} orc_key;

static int cmp_key(const void *a, const void *b) {
  const orc_key *x = (const orc_key *)a, *y = (const orc_key *)b;
  if (x->level != y->level) return x->level < y->level ? -1 : 1;
  if (x->prio != y->prio) return x->prio < y->prio ? -1 : 1;
  if (x->idx != y->idx) return x->idx < y->idx ? -1 : 1;
  return 0;
}

static int cmp_i64(const void *a, const void *b) {
  int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
  return x < y ? -1 : (x > y ? 1 : 0);
}

static int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }

#define ORC_NO_USE INT64_MAX

/* The paper's reclamation preference (Sec. 3.5): 1 when copy x should be
 * reclaimed before copy y.  red: resident on another device; dist: positions
 * until the next use on this device (ORC_NO_USE: none); load: reload time;
 * last: position of the last use on this device (-1: never used). */
static int paper_victim_before(int redx, int64_t distx, int64_t loadx, int64_t lastx,
                               int redy, int64_t disty, int64_t loady, int64_t lasty) {
  if (redx != redy) return redx > redy;                       /* redundant copies first */
  const int infx = distx == ORC_NO_USE || loadx == 0;         /* distance / reload cost */
  const int infy = disty == ORC_NO_USE || loady == 0;
  if (infx != infy) return infx > infy;
  if (!infx) {
    const int64_t a = distx * loady, b = disty * loadx;       /* distx/loadx vs disty/loady */
    if (a != b) return a > b;
  }
  return lastx < lasty;                                       /* least recently used */
}

/* ---------------------------------------------------------------------- */
/* scoring                                                                 */
/* ---------------------------------------------------------------------- */

/* The propagation of every plan; scores, the schedule rows and the ranking
 * keys (Eq. 12) are each written when their pointer is not NULL. */
/* Replica cap of one level: whether some model is held, as the level starts
 * (held) or by a load during it (loaded), on more devices than its cap. */
static int replica_over(const orc_window *w, const uint64_t *held, const uint64_t *loaded) {
  if (!w->replica_cap) return 0;
  for (int32_t m = 0; m < w->n_models; ++m) {
    int32_t copies = 0;
    for (int32_t d = 0; d < w->n_dev; ++d) copies += (int32_t)(((held[d] | loaded[d]) >> m) & 1u);
    if (copies > w->replica_cap[m]) return 1;
  }
  return 0;
}

static int simulate(const orc_window *w, const uint8_t *wf_class, const int8_t *dev,
                    const uint16_t *prio, const uint8_t *flags, int64_t n_plans,
                    orc_score *scores, int64_t *start_out, int64_t *finish_out,
                    int64_t *load_out, int32_t *peak_out, uint64_t *reclaim_out,
                    orc_phi *keys) {
  if (wf_class)
    for (int32_t f = 0; f < w->n_wf; ++f)
      if (wf_class[f] >= ORC_MAX_CLASSES) return ORC_ERR_CLASS;
  if (w->victim_order != ORC_VICTIM_REMAINING_LRU && w->victim_order != ORC_VICTIM_PAPER)
    return ORC_ERR_VICTIM;
  const int paper = w->victim_order == ORC_VICTIM_PAPER;
  if (w->dev_batch)
    for (int32_t d = 0; d < w->n_dev; ++d)
      if (w->dev_batch[d] < 1 || w->dev_batch[d] > ORC_MAX_BATCH) return ORC_ERR_BATCH;
  if (w->replica_cap && w->n_models >= 1 && w->n_models <= 64) {
    for (int32_t m = 0; m < w->n_models; ++m) {
      if (w->replica_cap[m] < 1) return ORC_ERR_REPLICA;
      int32_t copies = 0;
      for (int32_t d = 0; d < w->n_dev; ++d) copies += (int32_t)((w->init_resident[d] >> m) & 1u);
      if (copies > w->replica_cap[m]) return ORC_ERR_REPLICA;
    }
  }
  orc_struct st;
  int rc = build_struct(w, &st);
  if (rc) return rc;
  const int32_t N = w->n_act, D = w->n_dev, M = w->n_models, W = w->n_wf;
  const int32_t NB = (N + 3) / 4;
  size_t n = (size_t)(N > 0 ? N : 1);
  uint8_t *fuse = (uint8_t *)malloc(n), *pf = (uint8_t *)malloc(n), *member = (uint8_t *)malloc(n);
  int64_t *unit_Mx = (int64_t *)malloc(n * 8);
  orc_key *order = (orc_key *)malloc(n * sizeof(orc_key));
  int64_t *start = (int64_t *)malloc(n * 8), *finish = (int64_t *)malloc(n * 8),
          *load_start = (int64_t *)malloc(n * 8);
  int64_t *comp = (int64_t *)malloc((size_t)(W > 0 ? W : 1) * 8);
  /* per device and batch slot: free time, and the running unit's finish,
   * memory and model */
  const size_t ns = (size_t)D * ORC_MAX_BATCH;
  int64_t *slot_free = (int64_t *)malloc(ns * 8), *run_fin = (int64_t *)malloc(ns * 8),
          *run_mem = (int64_t *)malloc(ns * 8), *run_model = (int64_t *)malloc(ns * 8);
  int64_t *dispatched = (int64_t *)malloc((size_t)D * 8); /* last first-action time */
  int64_t *used = (int64_t *)malloc((size_t)D * 8),
          *peak = (int64_t *)malloc((size_t)D * 8);
  uint64_t *res = (uint64_t *)malloc((size_t)D * 8);
  uint64_t *reclaimed = (uint64_t *)malloc((size_t)D * 8);
  uint64_t *res_level = (uint64_t *)malloc((size_t)D * 8);
  uint64_t *loaded_level = (uint64_t *)malloc((size_t)D * 8);
  int64_t *dev_units = (int64_t *)malloc((size_t)D * 8);
  int64_t *next_after = (int64_t *)malloc(n * 8), *dev_index = (int64_t *)malloc(n * 8);
  int64_t *next_use = (int64_t *)malloc((size_t)D * M * 8);
  int64_t *remaining = (int64_t *)malloc((size_t)D * M * 8), *last = (int64_t *)malloc((size_t)D * M * 8);
  if (!fuse || !pf || !member || !unit_Mx || !order || !start || !finish ||
      !load_start || !comp || !slot_free || !run_fin || !run_mem || !run_model || !dispatched || !used || !peak || !res || !reclaimed || !remaining ||
      !last || !res_level || !loaded_level || !dev_units || !next_after || !dev_index || !next_use) {
    rc = ORC_ERR_NOMEM;
    goto done;
  }

  for (int64_t p = 0; p < n_plans; ++p) {
    const int8_t *pdev = dev + p * N;
    const uint16_t *pprio = prio + p * N;
    const uint8_t *pfl = flags + p * NB;
    orc_score sc;
    memset(&sc, 0, sizeof sc);

    /* ---- unit formation (Eq. 3, Eq. 4, Eq. 9) ---- */
    for (int32_t v = 0; v < N; ++v) {
      fuse[v] = (pfl[v / 4] >> (2 * (v % 4))) & 1u;
      pf[v] = (pfl[v / 4] >> (2 * (v % 4) + 1)) & 1u;
    }
    for (int32_t v = 0; v < N; ++v) member[v] = fuse[v] && st.fusible[v];
    int32_t n_units = 0;
    for (int32_t h = 0; h < N; ++h) {
      if (member[h]) continue;
      int32_t d = pdev[h];
      if (d < 0 || d >= D) {
        sc.status |= ORC_INELIGIBLE;
        continue;
      }
      int64_t Mx = 0;
      int32_t v = h;
      for (;;) {
        if (w->lat_us[(int64_t)v * D + d] < 0) sc.status |= ORC_INELIGIBLE;
        if (w->mem_mib[(int64_t)v * D + d] > Mx) Mx = w->mem_mib[(int64_t)v * D + d];
        int32_t c = st.child[v];
        if (c >= 0 && member[c]) v = c;
        else break;
      }
      unit_Mx[h] = Mx;
      order[n_units].level = st.level[h];
      order[n_units].prio = pprio[h];
      order[n_units].idx = h;
      ++n_units;
    }
    if (sc.status & ORC_INELIGIBLE) {
      sc.status = ORC_INELIGIBLE;
      if (scores) scores[p] = sc;
      if (keys) {
        memset(&keys[p], 0, sizeof keys[p]);
        keys[p].status = ORC_INELIGIBLE;
      }
      continue;
    }

    /* ---- resource order (Eq. 10; ready before near-ready, then priority) ---- */
    qsort(order, (size_t)n_units, sizeof(orc_key), cmp_key);
    for (int32_t i = 0; i < D * M; ++i) remaining[i] = 0;
    for (int32_t k = 0; k < n_units; ++k) {
      int32_t h = order[k].idx;
      remaining[pdev[h] * M + w->act_model[h]] += 1;
    }
    /* each unit's index among its device's units, the next use of the same
     * model on the same device after each unit (as such an index), and the
     * first use of every (device, model) */
    for (int32_t d = 0; d < D; ++d) dev_units[d] = 0;
    for (int32_t k = 0; k < n_units; ++k) dev_index[k] = dev_units[pdev[order[k].idx]]++;
    for (int32_t i = 0; i < D * M; ++i) next_use[i] = ORC_NO_USE;
    for (int32_t k = n_units - 1; k >= 0; --k) {
      int32_t h = order[k].idx;
      int64_t *nu = &next_use[pdev[h] * M + w->act_model[h]];
      next_after[k] = *nu;
      *nu = dev_index[k];
    }

    /* ---- pool snapshot ---- */
    for (int32_t d = 0; d < D; ++d) {
      dispatched[d] = w->dev_free0_us ? w->dev_free0_us[d] : 0;
      for (int32_t k = 0; k < ORC_MAX_BATCH; ++k) {
        slot_free[d * ORC_MAX_BATCH + k] = w->dev_free0_us ? w->dev_free0_us[d] : 0;
        run_fin[d * ORC_MAX_BATCH + k] = slot_free[d * ORC_MAX_BATCH + k];
        run_mem[d * ORC_MAX_BATCH + k] = 0;
        run_model[d * ORC_MAX_BATCH + k] = -1;
      }
      res[d] = w->init_resident[d];
      used[d] = 0;
      for (int32_t m = 0; m < M; ++m)
        if ((res[d] >> m) & 1u) used[d] += w->model_mib[m];
      peak[d] = used[d];
      for (int32_t m = 0; m < M; ++m) last[d * M + m] = -1;
      reclaimed[d] = 0;
    }
    int64_t n_loads = 0, n_evicts = 0;
    /* ranking-key terms (Eq. 12) */
    int64_t admitted[ORC_MAX_CLASSES] = {0, 0, 0, 0}, c_ready = 0, h_life = 0, timely = 0;

    /* copies reclaimed before each unit's first action (0 for members) */
    uint64_t *rec_row = reclaim_out ? reclaim_out + p * N : NULL;
    if (rec_row)
      for (int32_t i = 0; i < N; ++i) rec_row[i] = 0;

    /* ---- propagate units in resource order ---- */
    for (int32_t pos = 0; pos < n_units; ++pos) {
      int32_t h = order[pos].idx;
      int32_t d = pdev[h];
      int32_t m = w->act_model[h];
      int32_t wf = w->act_wf[h];
      int64_t Mx = unit_Mx[h];
      remaining[d * M + m] -= 1;
      /* pool residency as the unit's topological level starts; the replica
       * cap of the level that ends */
      if (pos == 0 || order[pos].level != order[pos - 1].level) {
        if (pos > 0 && replica_over(w, res_level, loaded_level)) sc.status |= ORC_REPLICA;
        for (int32_t e = 0; e < D; ++e) {
          res_level[e] = res[e];
          loaded_level[e] = 0;
        }
      }

      /* predicted release (Eq. 2): workflow arrival, or the latest
       * predecessor completion */
      int64_t r = w->wf_arrival_us[wf];
      for (int32_t k = w->pred_off[h]; k < w->pred_off[h + 1]; ++k)
        r = max64(r, finish[w->pred_idx[k]]);

      /* the device's slot that frees first (batch limit B; B = 1: the device) */
      const int32_t B = w->dev_batch ? w->dev_batch[d] : 1;
      int64_t *sf = &slot_free[d * ORC_MAX_BATCH];
      int32_t ks = 0;
      for (int32_t k = 1; k < B; ++k)
        if (sf[k] < sf[ks]) ks = k;
      const int64_t free_before = sf[ks];

      /* lifecycle (Eq. 5) with reclamation and the cumulative check (Eq. 11)
       * at the first action's time t: a load waits for the slot and starts
       * at the unit's release, or at the workflow's arrival when prefetched;
       * units still running at t hold their memory and lease their model */
      int miss = !((res[d] >> m) & 1u);
      int64_t need = (miss ? (int64_t)w->model_mib[m] : 0) + Mx;
      int64_t t = max64(max64(miss && pf[h] ? w->wf_arrival_us[wf] : r, free_before), dispatched[d]);
      int64_t run_act = 0;
      uint64_t leased = 0;
      for (;;) {
        int64_t next_fin = INT64_MAX;
        run_act = 0;
        leased = 0;
        for (int32_t k = 0; k < B; ++k) {
          const int32_t q = d * ORC_MAX_BATCH + k;
          if (run_fin[q] <= t) continue;
          run_act += run_mem[q];
          leased |= 1ull << run_model[q];
          if (run_fin[q] < next_fin) next_fin = run_fin[q];
        }
      while (used[d] + run_act + need > w->dev_cap_mib[d]) {
        uint64_t cand = res[d] & ~(1ull << m) & ~leased;
        if (!cand) break;
        int32_t victim = -1;
        for (int32_t m2 = 0; m2 < M; ++m2) {
          if (!((cand >> m2) & 1u)) continue;
          if (victim < 0) {
            victim = m2;
            continue;
          }
          if (paper) {
            int64_t key[2][4];
            const int32_t mm[2] = {m2, victim};
            for (int q = 0; q < 2; ++q) {
              int red = 0;
              for (int32_t e = 0; e < D; ++e)
                if (e != d && ((res_level[e] >> mm[q]) & 1u)) red = 1;
              const int64_t nu = next_use[d * M + mm[q]];
              key[q][0] = red;
              key[q][1] = nu == ORC_NO_USE ? ORC_NO_USE : nu - dev_index[pos];
              key[q][2] = w->load_us[mm[q] * D + d];
              key[q][3] = last[d * M + mm[q]];
            }
            if (paper_victim_before((int)key[0][0], key[0][1], key[0][2], key[0][3],
                                    (int)key[1][0], key[1][1], key[1][2], key[1][3]))
              victim = m2; /* equal keys keep the lower id (scanned first) */
            continue;
          }
          int alive2 = remaining[d * M + m2] > 0, aliveV = remaining[d * M + victim] > 0;
          if (alive2 != aliveV) {
            if (alive2 < aliveV) victim = m2;
          } else if (last[d * M + m2] < last[d * M + victim]) {
            victim = m2; /* equal keys keep the lower id (scanned first) */
          }
        }
        res[d] &= ~(1ull << victim);
        used[d] -= w->model_mib[victim];
        n_evicts += 1;
        reclaimed[d] |= 1ull << victim;
        if (rec_row) rec_row[h] |= 1ull << victim;
      }
        /* fits, or nothing left to wait for */
        if (!(used[d] + run_act + need > w->dev_cap_mib[d]) || next_fin == INT64_MAX) break;
        t = next_fin;
      }
      const int fits = !(used[d] + run_act + need > w->dev_cap_mib[d]);
      if (!fits) sc.status |= ORC_CAPACITY;

      /* ready work (F_t): no predecessor, and the workflow has arrived by
       * the window time 0 */
      const int ready = w->pred_off[h] == w->pred_off[h + 1] && w->wf_arrival_us[wf] <= 0;

      /* timeline (Eq. 7): a load waits for the device; it starts at the
       * unit's release, or at the workflow's arrival when prefetched */
      int64_t s;
      if (miss) {
        int64_t ls = t;
        int64_t le = ls + w->load_us[m * D + d];
        res[d] |= 1ull << m;
        loaded_level[d] |= 1ull << m;
        used[d] += w->model_mib[m];
        n_loads += 1;
        load_start[h] = ls;
        s = max64(r, le);
        /* reload of a copy this plan reclaimed from the device */
        if ((reclaimed[d] >> m) & 1u) h_life += le - ls;
        /* a prefetch is timely when its load is done by the release */
        if (!ready && pf[h] && le <= r) timely += 1;
        /* the delay a load adds to ready work */
        if (ready) h_life += s - max64(r, free_before);
      } else {
        load_start[h] = -1;
        s = t;
      }
      if (used[d] + run_act + Mx > peak[d]) peak[d] = used[d] + run_act + Mx;

      /* the unit's activations run back-to-back under one grant (Eq. 4) */
      int32_t v = h;
      for (;;) {
        start[v] = s;
        finish[v] = s + w->lat_us[(int64_t)v * D + d];
        s = finish[v];
        if (v != h) load_start[v] = -1;
        int32_t c = st.child[v];
        if (c >= 0 && member[c]) v = c;
        else break;
      }
      sf[ks] = s;
      dispatched[d] = t;
      run_fin[d * ORC_MAX_BATCH + ks] = s;
      run_mem[d * ORC_MAX_BATCH + ks] = Mx;
      run_model[d * ORC_MAX_BATCH + ks] = m;
      last[d * M + m] = pos;
      next_use[d * M + m] = next_after[pos];
      if (ready && fits) {
        admitted[wf_class ? wf_class[wf] : 0] += 1;
        c_ready = max64(c_ready, s);
      }
    }

    /* the replica cap of the last level */
    if (n_units > 0 && replica_over(w, res_level, loaded_level)) sc.status |= ORC_REPLICA;

    /* ---- reductions (Sec. 4 metrics) ---- */
    if (N > 0) {
      int64_t min_arr = w->wf_arrival_us[0], max_fin = finish[0];
      for (int32_t wf = 1; wf < W; ++wf)
        if (w->wf_arrival_us[wf] < min_arr) min_arr = w->wf_arrival_us[wf];
      for (int32_t i = 1; i < N; ++i) max_fin = max64(max_fin, finish[i]);
      sc.makespan_us = max_fin - min_arr;
      for (int32_t wf = 0; wf < W; ++wf) comp[wf] = INT64_MIN;
      for (int32_t i = 0; i < N; ++i) comp[w->act_wf[i]] = max64(comp[w->act_wf[i]], finish[i]);
      for (int32_t wf = 0; wf < W; ++wf) comp[wf] -= w->wf_arrival_us[wf];
      qsort(comp, (size_t)W, sizeof(int64_t), cmp_i64);
      int32_t k = (95 * W + 99) / 100; /* nearest rank: ceil(0.95 W) */
      sc.p95_us = comp[k - 1];
    }
    {
      float a = (float)sc.makespan_us;
      float b = (float)sc.p95_us;
      float x = w->w_makespan * a;
      float y = w->w_p95 * b;
      sc.objective = x + y;
    }
    int64_t headroom = (int64_t)w->dev_cap_mib[0] - peak[0];
    for (int32_t d = 1; d < D; ++d)
      if ((int64_t)w->dev_cap_mib[d] - peak[d] < headroom) headroom = (int64_t)w->dev_cap_mib[d] - peak[d];
    sc.min_headroom_mib = (int32_t)headroom;
    sc.n_loads = (uint16_t)(n_loads > 65535 ? 65535 : n_loads);
    sc.n_evicts = (uint16_t)(n_evicts > 65535 ? 65535 : n_evicts);
    if (scores) scores[p] = sc;
    if (keys) {
      orc_phi k;
      memset(&k, 0, sizeof k);
      k.c_ready_us = c_ready;
      k.h_life_us = h_life;
      for (int c = 0; c < ORC_MAX_CLASSES; ++c)
        k.admitted[c] = (uint16_t)(admitted[c] > 65535 ? 65535 : admitted[c]);
      k.timely_prefetch = (uint16_t)(timely > 65535 ? 65535 : timely);
      k.status = sc.status;
      keys[p] = k;
    }

    if (start_out) memcpy(start_out + p * N, start, (size_t)N * 8);
    if (finish_out) memcpy(finish_out + p * N, finish, (size_t)N * 8);
    if (load_out) memcpy(load_out + p * N, load_start, (size_t)N * 8);
    if (peak_out)
      for (int32_t d = 0; d < D; ++d) peak_out[p * D + d] = (int32_t)peak[d];
  }
  rc = ORC_OK;

done:
  free(fuse); free(pf); free(member); free(unit_Mx); free(order);
  free(start); free(finish); free(load_start); free(comp); free(slot_free); free(run_fin);
  free(run_mem); free(run_model); free(dispatched); free(used);
  free(peak); free(res); free(reclaimed); free(remaining); free(last);
  free(res_level); free(loaded_level); free(dev_units); free(next_after); free(dev_index); free(next_use);
  free_struct(&st);
  return rc;
}

int orc_score_plans(const orc_window *w, const int8_t *dev, const uint16_t *prio,
                    const uint8_t *flags, int64_t n_plans, orc_score *scores,
                    int64_t *start_out, int64_t *finish_out, int64_t *load_out,
                    int32_t *peak_out, uint64_t *reclaim_out) {
  return simulate(w, NULL, dev, prio, flags, n_plans, scores, start_out, finish_out, load_out,
                  peak_out, reclaim_out, NULL);
}

int orc_prefix(const orc_window *w, const int8_t *dev, const int64_t *start_us,
               const int64_t *finish_us, const int64_t *load_start_us,
               const uint64_t *reclaimed, uint8_t *commit, uint64_t *commit_reclaimed,
               int64_t *t_next_us) {
  const int32_t N = w->n_act, D = w->n_dev;
  for (int32_t i = 0; i < N; ++i)
    if (dev[i] < 0 || dev[i] >= D) return ORC_ERR_INDEX;
  /* the next predicted event after the window time 0: a unit's finish, a
   * load's end, a workflow's arrival */
  int64_t t = INT64_MAX;
  for (int32_t i = 0; i < N; ++i) {
    if (finish_us[i] > 0 && finish_us[i] < t) t = finish_us[i];
    if (load_start_us[i] >= 0) {
      const int64_t le = load_start_us[i] + w->load_us[(int64_t)w->act_model[i] * D + dev[i]];
      if (le > 0 && le < t) t = le;
    }
  }
  for (int32_t f = 0; f < w->n_wf; ++f)
    if (w->wf_arrival_us[f] > 0 && w->wf_arrival_us[f] < t) t = w->wf_arrival_us[f];
  *t_next_us = t;
  /* every action that begins before that event is committed now */
  for (int32_t i = 0; i < N; ++i) {
    const int grant = start_us[i] < t;
    const int load = load_start_us[i] >= 0 && load_start_us[i] < t;
    const int64_t first = load_start_us[i] >= 0 ? load_start_us[i] : start_us[i];
    commit[i] = (uint8_t)(grant | (load << 1));
    commit_reclaimed[i] = first < t ? reclaimed[i] : 0;
  }
  return ORC_OK;
}

int orc_phi_keys(const orc_window *w, const uint8_t *wf_class, const int8_t *dev,
                 const uint16_t *prio, const uint8_t *flags, int64_t n_plans, orc_phi *keys) {
  return simulate(w, wf_class, dev, prio, flags, n_plans, NULL, NULL, NULL, NULL, NULL, NULL, keys);
}

/* ---------------------------------------------------------------------- */
/* candidate generation                                                    */
/* ---------------------------------------------------------------------- */

void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * x0; /* multipliers of Philox-4x32 */
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * x2;
    const uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;
    const uint32_t y1 = (uint32_t)p1;
    const uint32_t y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
    const uint32_t y3 = (uint32_t)p0;
    x0 = y0;
    x1 = y1;
    x2 = y2;
    x3 = y3;
    k0 += 0x9E3779B9u; /* Weyl sequence: golden ratio and sqrt(3) - 1 */
    k1 += 0xBB67AE85u;
  }
  out[0] = x0;
  out[1] = x1;
  out[2] = x2;
  out[3] = x3;
}

/* floor(r * n / 2^32): a draw r scaled to [0, n) */
static uint32_t scale32(uint32_t r, uint32_t n) { return (uint32_t)(((uint64_t)r * n) >> 32); }

/* The rule tables of the candidate generator: each activation's best
 * binding (-1: none eligible), its earliest release, whether it is ready. */
static int rule_tables(const orc_window *w, int8_t *best, int64_t *rel_lb, uint8_t *ready) {
  const int32_t N = w->n_act, D = w->n_dev, M = w->n_models;
  int64_t *unlock = (int64_t *)calloc((size_t)M * D, 8);
  if (!unlock) return ORC_ERR_NOMEM;
  for (int32_t i = 0; i < N; ++i)
    ready[i] = w->pred_off[i] == w->pred_off[i + 1] && w->wf_arrival_us[w->act_wf[i]] <= 0;
  /* ready work a load of model m on device d would unlock */
  for (int32_t i = 0; i < N; ++i) {
    if (!ready[i]) continue;
    for (int32_t d = 0; d < D; ++d) {
      const int32_t l = w->lat_us[(int64_t)i * D + d];
      if (l >= 0) unlock[(int64_t)w->act_model[i] * D + d] += l;
    }
  }
  for (int32_t i = 0; i < N; ++i) {
    const int32_t m = w->act_model[i];
    int32_t b = -1, resident = 0;
    /* a resident accepting replica first: the fastest, then the lower id */
    for (int32_t d = 0; d < D; ++d) {
      const int32_t l = w->lat_us[(int64_t)i * D + d];
      if (l < 0 || !((w->init_resident[d] >> m) & 1u)) continue;
      if (!resident || l < w->lat_us[(int64_t)i * D + b]) b = d;
      resident = 1;
    }
    if (!resident) {
      /* otherwise the load worth the most: unlocked ready work per load time */
      for (int32_t d = 0; d < D; ++d) {
        const int32_t l = w->lat_us[(int64_t)i * D + d];
        if (l < 0) continue;
        if (b < 0) {
          b = d;
          continue;
        }
        const int64_t ld = w->load_us[(int64_t)m * D + d], lb = w->load_us[(int64_t)m * D + b];
        const int64_t ud = unlock[(int64_t)m * D + d], ub = unlock[(int64_t)m * D + b];
        int cmp; /* > 0: d is worth more than b */
        if ((ld == 0) != (lb == 0)) cmp = ld == 0 ? 1 : -1;
        else if (ld == 0) cmp = 0;
        else {
          const __int128 x = (__int128)ud * lb, y = (__int128)ub * ld;
          cmp = x > y ? 1 : (x < y ? -1 : 0);
        }
        if (cmp > 0 || (cmp == 0 && l < w->lat_us[(int64_t)i * D + b])) b = d;
      }
    }
    best[i] = (int8_t)b;
  }
  /* earliest release: predecessors on their fastest eligible devices */
  for (int32_t i = 0; i < N; ++i) {
    int64_t r = w->wf_arrival_us[w->act_wf[i]];
    for (int32_t k = w->pred_off[i]; k < w->pred_off[i + 1]; ++k) {
      const int32_t p = w->pred_idx[k];
      int64_t fast = -1;
      for (int32_t d = 0; d < D; ++d) {
        const int32_t l = w->lat_us[(int64_t)p * D + d];
        if (l >= 0 && (fast < 0 || l < fast)) fast = l;
      }
      if (rel_lb[p] + (fast < 0 ? 0 : fast) > r) r = rel_lb[p] + (fast < 0 ? 0 : fast);
    }
    rel_lb[i] = r;
  }
  free(unlock);
  return ORC_OK;
}

int orc_search_candidates(const orc_window *w, const int8_t *dev, const uint16_t *prio,
                          const uint8_t *flags, uint64_t seed, int32_t n_mut, int64_t first,
                          int64_t count, int32_t mode, int8_t *out_dev, uint16_t *out_prio,
                          uint8_t *out_flags) {
  if (mode != ORC_SEARCH_UNIFORM && mode != ORC_SEARCH_RULES) return ORC_ERR_SIZE;
  orc_struct st;
  int rc = build_struct(w, &st);
  if (rc) return rc;
  const int32_t N = w->n_act, D = w->n_dev, NB = (N + 3) / 4;
  const size_t n = (size_t)(N > 0 ? N : 1);
  int8_t *best = (int8_t *)malloc(n);
  int64_t *rel_lb = (int64_t *)malloc(n * 8);
  uint8_t *ready = (uint8_t *)malloc(n);
  if (!best || !rel_lb || !ready) {
    free(best);
    free(rel_lb);
    free(ready);
    free_struct(&st);
    return ORC_ERR_NOMEM;
  }
  if (mode == ORC_SEARCH_RULES) {
    rc = rule_tables(w, best, rel_lb, ready);
    if (rc) {
      free(best);
      free(rel_lb);
      free(ready);
      free_struct(&st);
      return rc;
    }
  }
  const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  for (int64_t k = 0; k < count; ++k) {
    int8_t *cd = out_dev + k * N;
    uint16_t *cp = out_prio + k * N;
    uint8_t *cf = out_flags + k * NB;
    memcpy(cd, dev, (size_t)N);
    memcpy(cp, prio, (size_t)N * 2);
    memcpy(cf, flags, (size_t)NB);
    if (N == 0) continue;
    const uint64_t c = (uint64_t)(first + k);
    for (int32_t t = 0; t < n_mut; ++t) {
      const uint32_t ctr[4] = {(uint32_t)c, (uint32_t)(c >> 32), (uint32_t)t, 0u};
      uint32_t r[4];
      orc_philox4x32_10(ctr, key, r);
      const int32_t i = (int32_t)scale32(r[1], (uint32_t)N);
      const uint32_t kind = r[0] >> 30;
      if (kind == 0 && mode == ORC_SEARCH_RULES) {
        /* BestFeasibleBinding */
        if (best[i] >= 0) cd[i] = best[i];
      } else if (kind == 0) {
        /* another eligible device (Eq. 8) */
        int32_t n_elig = 0;
        for (int32_t d = 0; d < D; ++d) n_elig += w->lat_us[(int64_t)i * D + d] >= 0;
        if (n_elig == 0) continue;
        int32_t pick = (int32_t)scale32(r[2], (uint32_t)n_elig);
        for (int32_t d = 0; d < D; ++d) {
          if (w->lat_us[(int64_t)i * D + d] < 0) continue;
          if (pick == 0) {
            cd[i] = (int8_t)d;
            break;
          }
          --pick;
        }
      } else if (kind == 1) {
        /* another order inside i's level (Eq. 10) */
        int32_t lo = i, hi = i + 1;
        while (lo > 0 && st.level[lo - 1] == st.level[i]) --lo;
        while (hi < N && st.level[hi] == st.level[i]) ++hi;
        const int32_t j = lo + (int32_t)scale32(r[2], (uint32_t)(hi - lo));
        const uint16_t tmp = cp[i];
        cp[i] = cp[j];
        cp[j] = tmp;
      } else if (kind == 2) {
        cf[i / 4] ^= (uint8_t)(1u << (2 * (i % 4)));     /* fuse bit (Eq. 3) */
      } else if (mode == ORC_SEARCH_RULES) {
        /* PlanPrefetch: near-ready work whose earliest release is within
         * the load time plus the dispatch slack */
        const int32_t d = cd[i];
        if (d < 0 || d >= D) continue;
        const int64_t ld = w->load_us[(int64_t)w->act_model[i] * D + d];
        const int on = !ready[i] && rel_lb[i] <= ld + w->prefetch_slack_us;
        const uint8_t bit = (uint8_t)(1u << (2 * (i % 4) + 1));
        cf[i / 4] = on ? (uint8_t)(cf[i / 4] | bit) : (uint8_t)(cf[i / 4] & ~bit);
      } else {
        cf[i / 4] ^= (uint8_t)(1u << (2 * (i % 4) + 1)); /* prefetch bit (Eq. 5) */
      }
    }
  }
  free(best);
  free(rel_lb);
  free(ready);
  free_struct(&st);
  return ORC_OK;
}
