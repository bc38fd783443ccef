/*
 * CPU oracle for eager multi-resolution substrate discovery (EMR-HyperNEAT, Phase 1).
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the benchmark's CPU-baseline
 * leg may load this library. It shares no code, header, table or helper with the HIP path.
 *
 * Plain, slow, obviously correct: double precision throughout (the paper does not fix a
 * precision), no blocking, no fusion, no reordering beyond the definitions it follows.
 *
 * What it computes, and where the paper defines it:
 *   - the multiresolution grid of cell centres (Section 3.1, Eq. 1), built by descending the
 *     quadtree from the root cell: a child's centre is its parent's centre +- half the child width;
 *   - one CPPN query per (genome, source, position) (Section 3.1, the batched query W); the CPPN is
 *     the raw genome evaluated in a topological order of its enabled edges (Section 2);
 *   - the variance of each cell's four children and the strict test var > theta (Section 3.2,
 *     Eq. 2 and the Superset Discovery theorem's proof);
 *   - three selection rules:
 *       PARENT : keep the children of every cell whose children's variance exceeds theta
 *                (the eager rule the superset proof describes);
 *       CHAIN  : additionally require every ancestor to pass (Eq. 2 read literally, with the root as
 *                the first gated cell);
 *       lazy   : ES-HyperNEAT's division phase (Section 2), a breadth-first subdivision that only
 *                expands cells whose children passed, implemented geometrically (centre, width) with
 *                no heap indices, so that it can be compared against the other two.
 *
 * Conventions (readings where the paper is silent):
 *   - depth D counts levels below the root: level l has 4^l cells of width 2/2^l, l = 1..D; the
 *     root (level 0, centre (0,0)) is the parent of level 1 and is never queried;
 *   - heap index: root F = 0, children of F are 4F+1+k, k = 0..3; bit 0 of k picks the +x half,
 *     bit 1 the +y half;
 *   - CPPN inputs are (x1, y1, x2, y2, 1); an outgoing source s puts s in (x1, y1) and the position
 *     in (x2, y2); an incoming source the other way round;
 *   - a non-input node computes act(bias + sum over enabled incoming edges of w * v_src), in edge-list
 *     order; activations: linear z, sigmoid 1/(1+e^-z), tanh z, gaussian e^(-z^2), sine sin z,
 *     abs |z|;
 *   - variance is the population variance (divide by 4) of the four children.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
  int32_t n_nodes, n_edges;
  const uint8_t* kind; /* 0..4 input roles x1,y1,x2,y2,bias; 5 hidden; 6 output */
  const uint8_t* act;
  const float* bias;   /* may be NULL (all zero) */
  const int32_t* src;
  const int32_t* dst;
  const float* w;
  const uint8_t* enabled; /* may be NULL (all enabled) */
} orc_genome;

typedef struct {
  float x, y;
  int32_t dir; /* 0 outgoing: CPPN(s, p); 1 incoming: CPPN(p, s) */
} orc_source;

enum { ORC_PARENT = 0, ORC_CHAIN = 1 };

/* ---------------------------------------------------------------- grid (Section 3.1, Eq. 1) */

/* Number of queried positions for depth D: the sum of the level sizes 4^l, l = 1..D. */
int64_t orc_n_positions(int depth) {
  int64_t n = 0, level_size = 1;
  for (int l = 1; l <= depth; ++l) {
    level_size *= 4;
    n += level_size;
  }
  return n;
}

/* Number of parent cells (levels 0..D-1) whose four children are queried. */
int64_t orc_n_parents(int depth) { return depth <= 0 ? 0 : 1 + orc_n_positions(depth - 1); }

/* Centre and level of heap cell F, by walking down from the root. */
void orc_cell(int64_t F, double* x, double* y, int* level) {
  int digits[40];
  int n = 0;
  while (F > 0) {
    digits[n++] = (int)((F - 1) % 4);
    F = (F - 1) / 4;
  }
  double cx = 0.0, cy = 0.0, half_width = 1.0; /* root: the square [-1,1]^2 */
  for (int t = n - 1; t >= 0; --t) {
    half_width *= 0.5; /* a child's half-width is half its parent's */
    cx += (digits[t] & 1) ? half_width : -half_width;
    cy += (digits[t] & 2) ? half_width : -half_width;
  }
  *x = cx;
  *y = cy;
  if (level) *level = n;
}

/* Centres of all queried positions, F = 1..N, as xy[2(F-1)], xy[2(F-1)+1]. */
void orc_grid(int depth, double* xy) {
  int64_t n = orc_n_positions(depth);
  for (int64_t p = 0; p < n; ++p) orc_cell(p + 1, &xy[2 * p], &xy[2 * p + 1], NULL);
}

/* ---------------------------------------------------------------- CPPN (Sections 2 and 3.1) */

double orc_act(int a, double z) {
  switch (a) {
    case 0: return z;                         /* linear */
    case 1: return 1.0 / (1.0 + exp(-z));     /* sigmoid */
    case 2: return tanh(z);                   /* tanh */
    case 3: return exp(-z * z);               /* gaussian */
    case 4: return sin(z);                    /* sine */
    case 5: return fabs(z);                   /* abs */
    default: return NAN;
  }
}

static int edge_on(const orc_genome* g, int e) { return g->enabled == NULL || g->enabled[e] != 0; }

/* Kahn's algorithm over the enabled edges. Writes a topological order of all nodes into order[]
 * and returns 0, or returns -1 if the enabled edges contain a cycle. */
int orc_topo_order(const orc_genome* g, int32_t* order) {
  int n = g->n_nodes;
  int* indeg = (int*)calloc((size_t)n, sizeof(int));
  int* queue = (int*)malloc((size_t)n * sizeof(int));
  for (int e = 0; e < g->n_edges; ++e)
    if (edge_on(g, e)) indeg[g->dst[e]]++;
  int head = 0, tail = 0;
  for (int v = 0; v < n; ++v)
    if (indeg[v] == 0) queue[tail++] = v;
  while (head < tail) {
    int u = queue[head++];
    for (int e = 0; e < g->n_edges; ++e) {
      if (!edge_on(g, e) || g->src[e] != u) continue;
      if (--indeg[g->dst[e]] == 0) queue[tail++] = g->dst[e];
    }
  }
  int ok = (tail == n);
  if (ok) memcpy(order, queue, (size_t)n * sizeof(int32_t));
  free(indeg);
  free(queue);
  return ok ? 0 : -1;
}

/* Evaluate the genome at inputs in[5] = (x1, y1, x2, y2, 1) following a topological order.
 * val[] is caller scratch of n_nodes doubles. Returns the output node's value. */
double orc_cppn(const orc_genome* g, const int32_t* order, const double in[5], double* val) {
  int out = -1;
  for (int t = 0; t < g->n_nodes; ++t) {
    int v = order[t];
    int k = g->kind[v];
    if (k <= 4) { /* an input node passes its role's value through */
      val[v] = in[k];
      continue;
    }
    double z = g->bias ? (double)g->bias[v] : 0.0;
    for (int e = 0; e < g->n_edges; ++e)
      if (edge_on(g, e) && g->dst[e] == v) z += (double)g->w[e] * val[g->src[e]];
    val[v] = orc_act(g->act[v], z);
    if (k == 6) out = v;
  }
  return out >= 0 ? val[out] : NAN;
}

/* CPPN query for source s at position (px, py) (Section 3.1 and Section 2's input tuple). */
static double query(const orc_genome* g, const int32_t* order, const orc_source* s, double px,
                    double py, double* val) {
  double in[5];
  if (s->dir == 0) {
    in[0] = s->x; in[1] = s->y; in[2] = px; in[3] = py;
  } else {
    in[0] = px; in[1] = py; in[2] = s->x; in[3] = s->y;
  }
  in[4] = 1.0;
  return orc_cppn(g, order, in, val);
}

/* Query the four children of parent P; returns their population variance (Section 3.2). */
static double parent_children(const orc_genome* g, const int32_t* order, const orc_source* s,
                              int64_t P, double w4[4], double* val) {
  for (int k = 0; k < 4; ++k) {
    double x, y;
    orc_cell(4 * P + 1 + k, &x, &y, NULL);
    w4[k] = query(g, order, s, x, y, val);
  }
  double mean = (w4[0] + w4[1] + w4[2] + w4[3]) / 4.0;
  double var = 0.0;
  for (int k = 0; k < 4; ++k) var += (w4[k] - mean) * (w4[k] - mean);
  return var / 4.0;
}

/* Evaluate given parents for one (genome, source): w4[4*i..], var[i]. Used for sampled checks. */
int orc_eval_parents(const orc_genome* g, const orc_source* s, const int64_t* parents, int64_t n,
                     double* w4, double* var) {
  int32_t* order = (int32_t*)malloc((size_t)g->n_nodes * sizeof(int32_t));
  double* val = (double*)malloc((size_t)g->n_nodes * sizeof(double));
  if (orc_topo_order(g, order) != 0) {
    free(order);
    free(val);
    return -1;
  }
  for (int64_t i = 0; i < n; ++i) var[i] = parent_children(g, order, s, parents[i], &w4[4 * i], val);
  free(order);
  free(val);
  return 0;
}

/* Evaluate the CPPN at arbitrary inputs: in5[5*i..5*i+4] -> out[i]. */
int orc_eval_points(const orc_genome* g, const double* in5, int64_t n, double* out) {
  int32_t* order = (int32_t*)malloc((size_t)g->n_nodes * sizeof(int32_t));
  double* val = (double*)malloc((size_t)g->n_nodes * sizeof(double));
  if (orc_topo_order(g, order) != 0) {
    free(order);
    free(val);
    return -1;
  }
  for (int64_t i = 0; i < n; ++i) out[i] = orc_cppn(g, order, &in5[5 * i], val);
  free(order);
  free(val);
  return 0;
}

/* ------------------------------------------------------- eager discovery (Section 3.2, Eq. 2) */

typedef struct {
  int64_t n, cap;
  int64_t* parent;
  double* w4;
  double* var;
} rec_buf;

static void rec_push(rec_buf* b, int64_t P, const double w4[4], double var) {
  if (b->n == b->cap) {
    b->cap = b->cap ? 2 * b->cap : 64;
    b->parent = (int64_t*)realloc(b->parent, (size_t)b->cap * sizeof(int64_t));
    b->w4 = (double*)realloc(b->w4, (size_t)b->cap * 4 * sizeof(double));
    b->var = (double*)realloc(b->var, (size_t)b->cap * sizeof(double));
  }
  b->parent[b->n] = P;
  memcpy(&b->w4[4 * b->n], w4, 4 * sizeof(double));
  b->var[b->n] = var;
  b->n++;
}

/* One (genome, source) pair: every parent in ascending heap order, kept by `mode`. */
static int discover_pair(const orc_genome* g, const orc_source* s, int depth, double theta, int mode,
                         rec_buf* out) {
  int32_t* order = (int32_t*)malloc((size_t)g->n_nodes * sizeof(int32_t));
  double* val = (double*)malloc((size_t)g->n_nodes * sizeof(double));
  if (orc_topo_order(g, order) != 0) {
    free(order);
    free(val);
    return -1;
  }
  int64_t Q = orc_n_parents(depth);
  unsigned char* pass = (mode == ORC_CHAIN) ? (unsigned char*)calloc((size_t)Q, 1) : NULL;
  for (int64_t P = 0; P < Q; ++P) {
    double w4[4];
    double var = parent_children(g, order, s, P, w4, val);
    int keep = var > theta;
    if (mode == ORC_CHAIN) {
      if (P > 0) keep = keep && pass[(P - 1) / 4];
      pass[P] = (unsigned char)keep;
    }
    if (keep) rec_push(out, P, w4, var);
  }
  free(pass);
  free(order);
  free(val);
  return 0;
}

/*
 * Whole population. Pairs are numbered genome-major: with src_offsets == NULL every genome uses the
 * n_shared sources (pair = g * n_shared + j); otherwise genome g uses sources
 * src_offsets[g] .. src_offsets[g+1]-1 (pair = that source index).
 * Outputs: pair_count[n_pairs]; records concatenated pair by pair in ascending parent order,
 * written only if the total fits in `capacity` (pass capacity 0 to count only).
 * Returns the total number of records, or -1 on a cyclic genome.
 */
int64_t orc_discover(const orc_genome* genomes, int32_t n_genomes, const orc_source* sources,
                     const int32_t* src_offsets, int32_t n_shared, int depth, double theta, int mode,
                     int64_t* pair_count, int64_t* parent, double* w4, double* var, int64_t capacity) {
  int64_t n_pairs = src_offsets ? src_offsets[n_genomes] : (int64_t)n_genomes * n_shared;
  rec_buf* bufs = (rec_buf*)calloc((size_t)(n_pairs > 0 ? n_pairs : 1), sizeof(rec_buf));
  int failed = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t pr = 0; pr < n_pairs; ++pr) {
    int64_t gi;
    if (src_offsets) {
      gi = 0;
      while (src_offsets[gi + 1] <= pr) gi++;
    } else {
      gi = pr / n_shared;
    }
    if (discover_pair(&genomes[gi], &sources[pr - (src_offsets ? 0 : gi * n_shared)], depth, theta,
                      mode, &bufs[pr]) != 0) {
#pragma omp atomic write
      failed = 1;
    }
  }
  int64_t total = 0;
  for (int64_t pr = 0; pr < n_pairs; ++pr) {
    pair_count[pr] = bufs[pr].n;
    total += bufs[pr].n;
  }
  if (!failed && total <= capacity) {
    int64_t at = 0;
    for (int64_t pr = 0; pr < n_pairs; ++pr) {
      rec_buf* b = &bufs[pr];
      if (b->n) {
        memcpy(&parent[at], b->parent, (size_t)b->n * sizeof(int64_t));
        memcpy(&w4[4 * at], b->w4, (size_t)b->n * 4 * sizeof(double));
        memcpy(&var[at], b->var, (size_t)b->n * sizeof(double));
      }
      at += b->n;
    }
  }
  for (int64_t pr = 0; pr < n_pairs; ++pr) {
    free(bufs[pr].parent);
    free(bufs[pr].w4);
    free(bufs[pr].var);
  }
  free(bufs);
  return failed ? -1 : total;
}

/* -------------------------------------------- lazy ES-HyperNEAT division phase (Section 2) */

/*
 * Breadth-first quadtree subdivision from the root cell (initial depth 0, no band pruning).
 * Every dequeued cell has its four children queried; if their variance exceeds theta the children
 * are "discovered" and, when they are above the maximum depth, queued for subdivision in turn.
 * Cells are handled purely geometrically (centre, half-width, level).
 * Outputs the discovered parents' centres cx, cy and levels (capacity entries at most) and
 * returns how many there were; n_queries receives the number of CPPN queries made.
 */
int64_t orc_lazy(const orc_genome* g, const orc_source* s, int depth, double theta, double* cx,
                 double* cy, int32_t* level, int64_t capacity, int64_t* n_queries) {
  int32_t* order = (int32_t*)malloc((size_t)g->n_nodes * sizeof(int32_t));
  double* val = (double*)malloc((size_t)g->n_nodes * sizeof(double));
  if (orc_topo_order(g, order) != 0) {
    free(order);
    free(val);
    return -1;
  }
  typedef struct { double x, y, half; int level; } cell;
  int64_t qcap = 1024, head = 0, tail = 0, found = 0, queries = 0;
  cell* queue = (cell*)malloc((size_t)qcap * sizeof(cell));
  queue[tail++] = (cell){0.0, 0.0, 1.0, 0};
  while (head < tail) {
    cell c = queue[head++];
    if (c.level >= depth) continue;
    double h = c.half * 0.5;
    cell kids[4];
    double w[4];
    for (int k = 0; k < 4; ++k) {
      kids[k] = (cell){c.x + ((k & 1) ? h : -h), c.y + ((k & 2) ? h : -h), h, c.level + 1};
      w[k] = query(g, order, s, kids[k].x, kids[k].y, val);
      queries++;
    }
    double mean = (w[0] + w[1] + w[2] + w[3]) / 4.0, var = 0.0;
    for (int k = 0; k < 4; ++k) var += (w[k] - mean) * (w[k] - mean);
    var /= 4.0;
    if (!(var > theta)) continue;
    if (found < capacity) {
      cx[found] = c.x;
      cy[found] = c.y;
      level[found] = c.level;
    }
    found++;
    if (c.level + 1 < depth) {
      for (int k = 0; k < 4; ++k) {
        if (tail == qcap) {
          /* compact the consumed head before growing */
          memmove(queue, queue + head, (size_t)(tail - head) * sizeof(cell));
          tail -= head;
          head = 0;
          if (tail == qcap) {
            qcap *= 2;
            queue = (cell*)realloc(queue, (size_t)qcap * sizeof(cell));
          }
        }
        queue[tail++] = kids[k];
      }
    }
  }
  free(queue);
  free(order);
  free(val);
  if (n_queries) *n_queries = queries;
  return found;
}

/* Harness control, no arithmetic: the OpenMP threads later calls may use (n >= 1). */
void orc_set_threads(int n) {
#ifdef _OPENMP
  if (n >= 1) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

int orc_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
