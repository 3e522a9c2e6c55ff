/*
 * mcf_oracle.c -- reference CPU solver for the layered min-cost max-flow
 * problem.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the plain, slow, obviously correct
 * oracle that the GPU library is checked against.  Only the test suite, the
 * package smoke check and the benchmark's CPU-baseline leg may load it; the
 * product path never does.  It shares no code, header or table with the GPU
 * library (it does not include the library's header), and it computes
 * everything in 64-bit integers.
 *
 * What it computes (paper Sec. V-A, Eq. 2, and Sec. IV: route as many
 * microbatches as possible, then at the least total delay): on the flow network
 *
 *     s0 -> s                     capacity supply,   cost 0
 *     s  -> in(0,i)               capacity infinite, cost src_cost[i]
 *     in(k,i) -> out(k,i)         capacity cap[k][i], cost node_cost[k][i]
 *     out(k,i) -> in(k+1,j)       capacity infinite, cost arc_cost[k][i][j]
 *                                 (absent when arc_cost == -1)
 *     out(S-1,i) -> t             capacity infinite, cost snk_cost[i]
 *
 * find an integral flow from s0 to t whose value F is maximum and whose cost
 * sum_e cost(e) * f(e) is minimum among flows of value F.  The data node of
 * the paper is both source and sink (Sec. V-A); it is split into the pair
 * (s, t) here, and s0 -> s caps the flow at the data node's supply of
 * microbatches.  A node's capacity (Sec. III: microbatches that fit in its
 * memory) is the capacity of its split arc in -> out, and Eq. 1's compute
 * halves (c_i + c_j) / 2 summed over a microbatch's closed route equal the
 * sum of the c_i of the nodes it visits, so each node's full compute cost
 * sits on its split arc.
 *
 * Method: successive shortest paths (Edmonds-Karp 1972, Tomizawa 1971) with
 * Johnson potentials.  All costs are >= 0, so pi = 0 is a valid start.  Each
 * round runs Dijkstra from s0 with a binary heap on the reduced costs
 * c(u,v) + pi(u) - pi(v) over arcs with residual capacity, stopping when t
 * is popped; then pi(v) += min(dist(v), dist(t)) for every v (unreached
 * vertices take dist(t)), the bottleneck delta along the shortest path is
 * pushed, F += delta and cost += delta * (pi(t) - pi(s0)).  The loop ends
 * when t is unreachable.  Each augmenting path's cost is also summed arc by
 * arc and compared with pi(t) - pi(s0) as a self-check.
 *
 * Vertex numbering (also the order of the exported potentials):
 *     0 = s0, 1 = s, 2 = t, 3 + 2*(k*n+i) = in(k,i), 4 + 2*(k*n+i) = out(k,i).
 *
 * Per-instance status: 0 ok, 1 bad input (negative capacity, cost or supply,
 * or an arc cost below -1), 99 internal self-check failure.
 */
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_INF_CAP ((int64_t)1 << 60)
#define OR_INF_DIST INT64_MAX
#define OR_NO_ARC (-1)

enum { OR_OK = 0, OR_BAD_INPUT = 1, OR_SELFCHECK = 99 };

typedef struct {
    int32_t S, n;
    const int32_t *cap, *ncost, *acost, *src, *snk; /* one instance */
    int32_t supply;
} or_instance;

typedef struct {
    int32_t V, E;           /* E counts both directions */
    int32_t *head;          /* [E] arc e goes tail(e) -> head[e] */
    int64_t *res;           /* [E] residual capacity */
    int64_t *cost;          /* [E] cost; cost[e ^ 1] == -cost[e] */
    int32_t *first;         /* [V+1] CSR over tails */
    int32_t *adj;           /* [E] arc ids grouped by tail */
    int32_t *tail;          /* [E] */
    /* original-arc ids for export (-1 when absent) */
    int32_t *id_split, *id_inter, *id_src, *id_snk;
} or_graph;

static int32_t v_in(int32_t n, int32_t k, int32_t i) { return 3 + 2 * (k * n + i); }
static int32_t v_out(int32_t n, int32_t k, int32_t i) { return 4 + 2 * (k * n + i); }

static int32_t add_arc(or_graph *g, int32_t u, int32_t v, int64_t cap, int64_t c)
{
    int32_t e = g->E;
    g->tail[e] = u; g->head[e] = v; g->res[e] = cap; g->cost[e] = c;
    g->tail[e + 1] = v; g->head[e + 1] = u; g->res[e + 1] = 0; g->cost[e + 1] = -c;
    g->E += 2;
    return e;
}

static void graph_free(or_graph *g)
{
    free(g->head); free(g->res); free(g->cost); free(g->first); free(g->adj);
    free(g->tail); free(g->id_split); free(g->id_inter); free(g->id_src); free(g->id_snk);
}

static int graph_build(or_graph *g, const or_instance *in)
{
    int32_t S = in->S, n = in->n;
    int64_t inter = (int64_t)(S > 1 ? S - 1 : 0) * n * n;
    int64_t emax = 2 * (1 + n + (int64_t)S * n + inter + n);
    memset(g, 0, sizeof(*g));
    g->V = 3 + 2 * S * n;
    g->head = malloc(sizeof(int32_t) * emax);
    g->res = malloc(sizeof(int64_t) * emax);
    g->cost = malloc(sizeof(int64_t) * emax);
    g->tail = malloc(sizeof(int32_t) * emax);
    g->adj = malloc(sizeof(int32_t) * emax);
    g->first = calloc((size_t)g->V + 1, sizeof(int32_t));
    g->id_split = malloc(sizeof(int32_t) * (size_t)S * n);
    g->id_inter = malloc(sizeof(int32_t) * (size_t)(inter > 0 ? inter : 1));
    g->id_src = malloc(sizeof(int32_t) * n);
    g->id_snk = malloc(sizeof(int32_t) * n);
    if (!g->head || !g->res || !g->cost || !g->tail || !g->adj || !g->first ||
        !g->id_split || !g->id_inter || !g->id_src || !g->id_snk)
        return -1;

    add_arc(g, 0, 1, in->supply, 0);
    for (int32_t i = 0; i < n; i++)
        g->id_src[i] = add_arc(g, 1, v_in(n, 0, i), OR_INF_CAP, in->src[i]);
    for (int32_t k = 0; k < S; k++)
        for (int32_t i = 0; i < n; i++)
            g->id_split[k * n + i] = add_arc(g, v_in(n, k, i), v_out(n, k, i),
                                             in->cap[k * n + i], in->ncost[k * n + i]);
    for (int32_t k = 0; k + 1 < S; k++)
        for (int32_t i = 0; i < n; i++)
            for (int32_t j = 0; j < n; j++) {
                int64_t q = ((int64_t)k * n + i) * n + j;
                int32_t a = in->acost[q];
                g->id_inter[q] = (a == OR_NO_ARC) ? -1
                    : add_arc(g, v_out(n, k, i), v_in(n, k + 1, j), OR_INF_CAP, a);
            }
    for (int32_t i = 0; i < n; i++)
        g->id_snk[i] = add_arc(g, v_out(n, S - 1, i), 2, OR_INF_CAP, in->snk[i]);

    /* CSR of arc ids by tail vertex */
    for (int32_t e = 0; e < g->E; e++) g->first[g->tail[e] + 1]++;
    for (int32_t v = 0; v < g->V; v++) g->first[v + 1] += g->first[v];
    int32_t *fill = malloc(sizeof(int32_t) * g->V);
    if (!fill) return -1;
    memcpy(fill, g->first, sizeof(int32_t) * g->V);
    for (int32_t e = 0; e < g->E; e++) g->adj[fill[g->tail[e]]++] = e;
    free(fill);
    return 0;
}

/* ---- binary min-heap of (key, vertex) with lazy deletion ---- */
typedef struct { int64_t key; int32_t v; } or_item;
typedef struct { or_item *a; int64_t size; } or_heap;

static void heap_push(or_heap *h, int64_t key, int32_t v)
{
    int64_t i = h->size++;
    h->a[i].key = key; h->a[i].v = v;
    while (i > 0) {
        int64_t p = (i - 1) / 2;
        if (h->a[p].key <= h->a[i].key) break;
        or_item t = h->a[p]; h->a[p] = h->a[i]; h->a[i] = t;
        i = p;
    }
}

static or_item heap_pop(or_heap *h)
{
    or_item top = h->a[0];
    h->a[0] = h->a[--h->size];
    int64_t i = 0;
    for (;;) {
        int64_t l = 2 * i + 1, r = l + 1, m = i;
        if (l < h->size && h->a[l].key < h->a[m].key) m = l;
        if (r < h->size && h->a[r].key < h->a[m].key) m = r;
        if (m == i) break;
        or_item t = h->a[m]; h->a[m] = h->a[i]; h->a[i] = t;
        i = m;
    }
    return top;
}

static int instance_valid(const or_instance *in)
{
    int32_t S = in->S, n = in->n;
    if (in->supply < 0) return 0;
    for (int64_t q = 0; q < (int64_t)S * n; q++)
        if (in->cap[q] < 0 || in->ncost[q] < 0) return 0;
    for (int32_t i = 0; i < n; i++)
        if (in->src[i] < 0 || in->snk[i] < 0) return 0;
    for (int64_t q = 0; q < (int64_t)(S - 1) * n * n; q++)
        if (in->acost[q] < OR_NO_ARC) return 0;
    return 1;
}

typedef struct {
    int64_t F, cost, augmentations, arc_scans;
    int32_t status;
} or_result;

/* Solves one instance.  Output arrays (any may be NULL) use the canonical
 * per-instance layout: node_flow[S][n], arc_flow[S-1][n][n], src_flow[n],
 * snk_flow[n], potential[V]. */
static or_result solve_one(const or_instance *in, int32_t *node_flow, int32_t *arc_flow,
                           int32_t *src_flow, int32_t *snk_flow, int64_t *potential)
{
    or_result r = {0, 0, 0, 0, OR_OK};
    int32_t S = in->S, n = in->n;
    if (!instance_valid(in)) {
        r.status = OR_BAD_INPUT;
    }
    or_graph g;
    if (graph_build(&g, in) != 0) { graph_free(&g); r.status = OR_SELFCHECK; return r; }
    int32_t V = g.V;
    int64_t *pi = calloc(V, sizeof(int64_t));
    int64_t *dist = malloc(sizeof(int64_t) * V);
    int32_t *pred = malloc(sizeof(int32_t) * V);
    char *done = malloc(V);
    or_heap h;
    h.a = malloc(sizeof(or_item) * ((int64_t)g.E + 2));
    h.size = 0;

    while (r.status == OR_OK) {
        for (int32_t v = 0; v < V; v++) { dist[v] = OR_INF_DIST; pred[v] = -1; done[v] = 0; }
        dist[0] = 0;
        h.size = 0;
        heap_push(&h, 0, 0);
        while (h.size > 0) {
            or_item it = heap_pop(&h);
            int32_t u = it.v;
            if (done[u] || it.key != dist[u]) continue;
            done[u] = 1;
            if (u == 2) break;                      /* t settled */
            for (int32_t p = g.first[u]; p < g.first[u + 1]; p++) {
                int32_t e = g.adj[p];
                r.arc_scans++;
                if (g.res[e] <= 0) continue;
                int32_t v = g.head[e];
                int64_t rc = g.cost[e] + pi[u] - pi[v];
                if (rc < 0) { r.status = OR_SELFCHECK; break; }
                int64_t nd = dist[u] + rc;
                if (nd < dist[v]) {
                    dist[v] = nd; pred[v] = e;
                    heap_push(&h, nd, v);
                }
            }
        }
        if (r.status != OR_OK || dist[2] == OR_INF_DIST) break;
        int64_t dt = dist[2];
        for (int32_t v = 0; v < V; v++) pi[v] += (dist[v] < dt) ? dist[v] : dt;

        int64_t delta = OR_INF_CAP, pathcost = 0;
        for (int32_t v = 2; v != 0; v = g.tail[pred[v]]) {
            int32_t e = pred[v];
            if (g.res[e] < delta) delta = g.res[e];
            pathcost += g.cost[e];
        }
        if (pathcost != pi[2] - pi[0] || delta <= 0) { r.status = OR_SELFCHECK; break; }
        for (int32_t v = 2; v != 0; v = g.tail[pred[v]]) {
            int32_t e = pred[v];
            g.res[e] -= delta;
            g.res[e ^ 1] += delta;
        }
        r.F += delta;
        r.cost += delta * (pi[2] - pi[0]);
        r.augmentations++;
    }

    if (r.status == OR_OK) {
        /* the flow on an original arc is the residual of its reverse arc */
        if (node_flow)
            for (int64_t q = 0; q < (int64_t)S * n; q++) node_flow[q] = (int32_t)g.res[g.id_split[q] ^ 1];
        if (arc_flow)
            for (int64_t q = 0; q < (int64_t)(S - 1) * n * n; q++)
                arc_flow[q] = g.id_inter[q] < 0 ? 0 : (int32_t)g.res[g.id_inter[q] ^ 1];
        if (src_flow) for (int32_t i = 0; i < n; i++) src_flow[i] = (int32_t)g.res[g.id_src[i] ^ 1];
        if (snk_flow) for (int32_t i = 0; i < n; i++) snk_flow[i] = (int32_t)g.res[g.id_snk[i] ^ 1];
        if (potential) memcpy(potential, pi, sizeof(int64_t) * V);
    } else {
        r.F = 0; r.cost = 0;
        if (node_flow) memset(node_flow, 0, sizeof(int32_t) * S * n);
        if (arc_flow) memset(arc_flow, 0, sizeof(int32_t) * (size_t)(S - 1) * n * n);
        if (src_flow) memset(src_flow, 0, sizeof(int32_t) * n);
        if (snk_flow) memset(snk_flow, 0, sizeof(int32_t) * n);
        if (potential) memset(potential, 0, sizeof(int64_t) * V);
    }
    free(pi); free(dist); free(pred); free(done); free(h.a);
    graph_free(&g);
    return r;
}

/* ---- batch driver with a pthread pool over instances ---- */
typedef struct {
    int32_t B, S, n;
    const int32_t *cap, *ncost, *acost, *src, *snk, *supply;
    int64_t *F, *cost, *stats;
    int32_t *status, *node_flow, *arc_flow, *src_flow, *snk_flow;
    int64_t *potential;
    int32_t next;            /* shared work counter */
    int32_t *zeros;          /* [n] for NULL src/snk */
} or_job;

static void *worker(void *arg)
{
    or_job *jb = (or_job *)arg;
    int32_t S = jb->S, n = jb->n, V = 3 + 2 * S * n;
    int64_t sn = (int64_t)S * n, ann = (int64_t)(S > 1 ? S - 1 : 0) * n * n;
    for (;;) {
        int32_t b = __atomic_fetch_add(&jb->next, 1, __ATOMIC_RELAXED);
        if (b >= jb->B) break;
        or_instance in;
        in.S = S; in.n = n;
        in.cap = jb->cap + b * sn;
        in.ncost = jb->ncost + b * sn;
        in.acost = jb->acost ? jb->acost + b * ann : NULL;
        in.src = jb->src ? jb->src + (int64_t)b * n : jb->zeros;
        in.snk = jb->snk ? jb->snk + (int64_t)b * n : jb->zeros;
        in.supply = jb->supply[b];
        or_result r = solve_one(&in,
            jb->node_flow ? jb->node_flow + b * sn : NULL,
            jb->arc_flow ? jb->arc_flow + b * ann : NULL,
            jb->src_flow ? jb->src_flow + (int64_t)b * n : NULL,
            jb->snk_flow ? jb->snk_flow + (int64_t)b * n : NULL,
            jb->potential ? jb->potential + (int64_t)b * V : NULL);
        if (jb->F) jb->F[b] = r.F;
        if (jb->cost) jb->cost[b] = r.cost;
        if (jb->status) jb->status[b] = r.status;
        if (jb->stats) { jb->stats[2 * b] = r.augmentations; jb->stats[2 * b + 1] = r.arc_scans; }
    }
    return NULL;
}

/* Solves B independent instances laid out as documented in the header
 * comment above (int32 inputs, batch-major).  src_cost / snk_cost may be
 * NULL (all zero); arc_cost must be non-NULL when S > 1.  Outputs may be
 * NULL.  stats, if given, receives [B][2] = (augmentations, arc scans).
 * Returns the number of threads used, or -1 on a bad shape. */
int oracle_solve_batch(int32_t B, int32_t S, int32_t n,
                       const int32_t *node_cap, const int32_t *node_cost, const int32_t *arc_cost,
                       const int32_t *src_cost, const int32_t *snk_cost, const int32_t *supply,
                       int64_t *flow_value, int64_t *total_cost, int32_t *status,
                       int32_t *node_flow, int32_t *arc_flow, int32_t *src_flow, int32_t *snk_flow,
                       int64_t *potential, int64_t *stats, int32_t nthreads)
{
    if (B < 0 || S < 1 || n < 1 || !node_cap || !node_cost || !supply) return -1;
    if (S > 1 && !arc_cost) return -1;
    or_job jb;
    memset(&jb, 0, sizeof(jb));
    jb.B = B; jb.S = S; jb.n = n;
    jb.cap = node_cap; jb.ncost = node_cost; jb.acost = arc_cost;
    jb.src = src_cost; jb.snk = snk_cost; jb.supply = supply;
    jb.F = flow_value; jb.cost = total_cost; jb.status = status; jb.stats = stats;
    jb.node_flow = node_flow; jb.arc_flow = arc_flow; jb.src_flow = src_flow;
    jb.snk_flow = snk_flow; jb.potential = potential;
    jb.zeros = calloc(n, sizeof(int32_t));
    if (!jb.zeros) return -1;
    if (nthreads < 1) nthreads = 1;
    if (nthreads > B) nthreads = B > 0 ? B : 1;
    pthread_t *th = malloc(sizeof(pthread_t) * nthreads);
    int32_t started = 0;
    for (int32_t t = 1; t < nthreads; t++)
        if (pthread_create(&th[t], NULL, worker, &jb) == 0) started++; else break;
    worker(&jb);
    for (int32_t t = 1; t <= started; t++) pthread_join(th[t], NULL);
    free(th);
    free(jb.zeros);
    return started + 1;
}
