/*
 * oracle_check.c -- drives the C oracle (oracle/pardnn_oracle.c) under
 * AddressSanitizer and UndefinedBehaviorSanitizer: seeded random DAGs of
 * 0..60 nodes with multi-edges, the degenerate graphs (empty, no edges, one
 * chain) and every documented error (cycle, self-loop, id out of range,
 * negative weight, int64 overflow, NULL arrays). On each valid graph it
 * checks the definitions the oracle claims (Table 2: tl and bl relax every
 * edge and are attained; M = max tl + bl; the path is critical, starts at a
 * source, ends at a sink, and steps along tight edges; levels increase along
 * every edge; label sums add up to the total memory). Exit status 0 when all
 * hold; a sanitizer finding aborts.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "pardnn_oracle.h"

static int n_failed = 0;

#define EXPECT(cond)                                                         \
    do {                                                                     \
        if (!(cond)) {                                                       \
            fprintf(stderr, "check failed (line %d): %s\n", __LINE__, #cond); \
            n_failed++;                                                      \
        }                                                                    \
    } while (0)

/* splitmix64: the seeded source of every input here */
static uint64_t rng_state;
static uint64_t next_u64(void)
{
    uint64_t z = (rng_state += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}
static int64_t below(int64_t n) { return n > 0 ? (int64_t)(next_u64() % (uint64_t)n) : 0; }

static int64_t cost_of(const int32_t *lab, const int32_t *src, const int32_t *dst,
                       const int64_t *cost, int64_t e)
{
    return lab[src[e]] == lab[dst[e]] ? 0 : cost[e];
}

static void check_graph(int32_t V, int64_t E, const int32_t *src, const int32_t *dst,
                        const int64_t *comp, const int64_t *cost, const int64_t *mem,
                        const int32_t *lab, int32_t K)
{
    int32_t *level = malloc(sizeof(int32_t) * (V + 1));
    int32_t *order = malloc(sizeof(int32_t) * (V + 1));
    int32_t *lptr = malloc(sizeof(int32_t) * (V + 2));
    int64_t *tl = malloc(sizeof(int64_t) * (V + 1));
    int64_t *bl = malloc(sizeof(int64_t) * (V + 1));
    uint8_t *crit = malloc(V + 1);
    int32_t *path = malloc(sizeof(int32_t) * (V + 1));
    int64_t *lm = malloc(sizeof(int64_t) * K);
    int64_t *ov = malloc(sizeof(int64_t) * K);
    int64_t *cap = malloc(sizeof(int64_t) * K);
    int32_t nl = -1, plen = -1;
    int64_t M = -1;

    EXPECT(orc_validate(V, E, src, dst, comp, cost, mem) == ORC_OK);
    EXPECT(orc_levelize(V, E, src, dst, level, order, lptr, &nl) == ORC_OK);
    EXPECT(nl >= (V > 0) && nl <= V && lptr[0] == 0 && lptr[nl] == V);
    for (int32_t l = 0; l < nl; l++) EXPECT(lptr[l] < lptr[l + 1]);
    for (int64_t e = 0; e < E; e++) EXPECT(level[dst[e]] > level[src[e]]);
    EXPECT(orc_tb_levels(V, E, src, dst, comp, cost, lab, tl, bl, &M) == ORC_OK);
    int64_t m = 0;
    for (int32_t v = 0; v < V; v++) m = tl[v] + bl[v] > m ? tl[v] + bl[v] : m;
    EXPECT(M == m);
    /* relaxed on every edge, and attained (by an edge, or as the empty max) */
    for (int64_t e = 0; e < E; e++) {
        const int64_t c = cost_of(lab, src, dst, cost, e);
        EXPECT(tl[dst[e]] >= tl[src[e]] + comp[src[e]] + c);
        EXPECT(bl[src[e]] >= comp[src[e]] + c + bl[dst[e]]);
    }
    for (int32_t v = 0; v < V; v++) {
        int t_ok = tl[v] == 0, b_ok = bl[v] == comp[v];
        for (int64_t e = 0; e < E; e++) {
            const int64_t c = cost_of(lab, src, dst, cost, e);
            if (dst[e] == v && tl[v] == tl[src[e]] + comp[src[e]] + c) t_ok = 1;
            if (src[e] == v && bl[v] == comp[v] + c + bl[dst[e]]) b_ok = 1;
        }
        EXPECT(t_ok && b_ok);
    }
    EXPECT(orc_critical_path(V, E, src, dst, comp, cost, lab, tl, bl, M, crit, path, &plen) ==
           ORC_OK);
    for (int32_t v = 0; v < V; v++) EXPECT(crit[v] == (tl[v] + bl[v] == M));
    EXPECT(plen >= (V > 0) && plen <= V);
    if (plen > 0) {
        EXPECT(tl[path[0]] == 0);
        int64_t len = 0;
        for (int32_t i = 0; i < plen; i++) {
            EXPECT(crit[path[i]]);
            len += comp[path[i]];
            if (i + 1 < plen) {
                int64_t best = -1;
                for (int64_t e = 0; e < E; e++)
                    if (src[e] == path[i] && dst[e] == path[i + 1]) {
                        const int64_t c = cost_of(lab, src, dst, cost, e);
                        best = c > best ? c : best;
                    }
                EXPECT(best >= 0);
                len += best;
            }
        }
        for (int64_t e = 0; e < E; e++) EXPECT(src[e] != path[plen - 1]);
        EXPECT(len == M);
    }
    for (int32_t k = 0; k < K; k++) cap[k] = (int64_t)below(200);
    EXPECT(orc_label_memory(V, mem, lab, K, cap, lm, ov) == ORC_OK);
    int64_t tot = 0, want = 0;
    for (int32_t k = 0; k < K; k++) {
        tot += lm[k];
        EXPECT(ov[k] == (lm[k] > cap[k] ? lm[k] - cap[k] : 0));
    }
    for (int32_t v = 0; v < V; v++) want += mem[v];
    EXPECT(tot == want);
    free(level); free(order); free(lptr); free(tl); free(bl); free(crit); free(path);
    free(lm); free(ov); free(cap);
}

int main(void)
{
    rng_state = 20080863ull;
    /* random DAGs: edges go from lower to higher rank of a random order */
    for (int it = 0; it < 400; it++) {
        const int32_t V = (int32_t)below(61);
        const int64_t E = V > 1 ? below(4 * (int64_t)V) : 0;
        const int32_t K = 1 + (int32_t)below(5);
        int32_t *perm = malloc(sizeof(int32_t) * (V + 1));
        int32_t *src = malloc(sizeof(int32_t) * (E + 1));
        int32_t *dst = malloc(sizeof(int32_t) * (E + 1));
        int64_t *comp = malloc(sizeof(int64_t) * (V + 1));
        int64_t *mem = malloc(sizeof(int64_t) * (V + 1));
        int64_t *cost = malloc(sizeof(int64_t) * (E + 1));
        int32_t *lab = malloc(sizeof(int32_t) * (V + 1));
        for (int32_t v = 0; v < V; v++) perm[v] = v;
        for (int32_t v = V - 1; v > 0; v--) {
            const int32_t j = (int32_t)below(v + 1), t = perm[v];
            perm[v] = perm[j];
            perm[j] = t;
        }
        for (int64_t e = 0; e < E; e++) {
            int32_t a = (int32_t)below(V), b = (int32_t)below(V);
            if (a == b) b = (a + 1) % V;
            if (a > b) { const int32_t t = a; a = b; b = t; }
            src[e] = perm[a];
            dst[e] = perm[b];
            cost[e] = below(4) == 0 ? 0 : below(50);
        }
        for (int32_t v = 0; v < V; v++) {
            comp[v] = below(3) == 0 ? 0 : below(40);
            mem[v] = below(100);
            lab[v] = (int32_t)below(K);
        }
        check_graph(V, E, src, dst, comp, cost, mem, lab, K);
        free(perm); free(src); free(dst); free(comp); free(mem); free(cost); free(lab);
    }

    /* a chain 0 -> 1 -> ... -> 9 on two alternating labels */
    {
        int32_t src[9], dst[9], lab[10];
        int64_t comp[10], mem[10], cost[9];
        for (int i = 0; i < 10; i++) { comp[i] = i + 1; mem[i] = 1; lab[i] = i % 2; }
        for (int i = 0; i < 9; i++) { src[i] = i; dst[i] = i + 1; cost[i] = 2; }
        check_graph(10, 9, src, dst, comp, cost, mem, lab, 2);
    }

    /* errors */
    {
        int32_t src[3] = {0, 1, 2}, dst[3] = {1, 2, 0};
        int64_t w[3] = {1, 1, 1}, neg[3] = {1, -1, 1}, big[3] = {INT64_MAX, 1, 0};
        int32_t lvl[4], ord[4], lp[5], nl = 0;
        EXPECT(orc_levelize(3, 3, src, dst, lvl, ord, lp, &nl) == ORC_E_CYCLE);
        int32_t s1[1] = {1}, d1[1] = {1};
        EXPECT(orc_levelize(3, 1, s1, d1, lvl, ord, lp, &nl) == ORC_E_CYCLE);
        int32_t s2[1] = {0}, d2[1] = {3};
        EXPECT(orc_validate(3, 1, s2, d2, w, w, w) == ORC_E_INVAL);
        EXPECT(orc_levelize(3, 1, s2, d2, lvl, ord, lp, &nl) == ORC_E_INVAL);
        EXPECT(orc_validate(3, 2, src, dst, neg, w, w) == ORC_E_INVAL);
        EXPECT(orc_validate(3, 2, src, dst, w, neg, w) == ORC_E_INVAL);
        EXPECT(orc_validate(3, 2, src, dst, w, w, neg) == ORC_E_INVAL);
        EXPECT(orc_validate(3, 2, src, dst, big, w, w) == ORC_E_OVERFLOW);
        EXPECT(orc_validate(3, 2, src, dst, w, w, big) == ORC_E_OVERFLOW);
        EXPECT(orc_validate(3, 2, NULL, dst, w, w, w) == ORC_E_INVAL);
        EXPECT(orc_validate(3, 0, NULL, NULL, NULL, NULL, w) == ORC_E_INVAL);
        EXPECT(orc_validate(-1, 0, NULL, NULL, NULL, NULL, NULL) == ORC_E_INVAL);
    }

    if (n_failed) fprintf(stderr, "%d check(s) failed\n", n_failed);
    else printf("oracle checks: all passed\n");
    return n_failed ? 1 : 0;
}
