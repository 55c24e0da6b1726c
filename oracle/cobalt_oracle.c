/*
 * Oracle for the co-activation token-routing path of Cobalt
 * ("Leveraging Expert Co-activation for Efficient Distributed MoE Training").
 *
 * TEST INFRASTRUCTURE ONLY. This is a plain, slow, single-threaded C
 * statement of what the routing path computes, used to check the HIP
 * library. Only the test suite, the smoke check and the benchmark's CPU
 * baseline leg may load it. It shares no source, header, table or helper
 * with the HIP library; the two agree only through the definitions below.
 *
 * Every loop runs in index order; nothing is blocked, fused or reordered.
 *
 * Pins (what checks this file against something other than itself) are in
 * tests/test_oracle_*.py. One part is "parity unpinned" by the paper: WHICH
 * replica RandomNode / UniformChoice return (Algorithm 1 only says the
 * choice is random, and uniform for ranks). The counter-based draw below is
 * this implementation's reading, pinned by SplitMix64's published outputs
 * and by uniformity tests, not by any value in the paper.
 *
 * Notation (Section 3.1): T tokens, E experts, K selections per token,
 * N nodes of g ranks, G = N*g ranks, node(r) = r / g. Pair p = t*K + j is
 * slot j of token t.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define REF_OK 0
#define REF_EINVAL 1
#define REF_EDATA 5

/* ---------------------------------------------------------------------- */
/* SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom number   */
/* generators", OOPSLA 2014): the generator advances its state by the      */
/* golden-ratio increment 0x9e3779b97f4a7c15 and returns a mix of the new  */
/* state. ref_splitmix64(z) is the output produced from state z.           */
/* ---------------------------------------------------------------------- */
uint64_t ref_splitmix64(uint64_t z)
{
    z += 0x9e3779b97f4a7c15ULL;
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

/* Key of one (seed, step): every draw of that step hashes the pair index
 * with it. */
uint64_t ref_rng_key(uint64_t seed, uint64_t step)
{
    return ref_splitmix64(ref_splitmix64(seed) ^ step);
}

/* Uniform index in [0, cnt) for pair p and draw stream s (0 = node,
 * 1 = rank): the high 32 bits of the hash scaled by cnt (multiply-shift
 * range reduction, Lemire 2019). */
uint32_t ref_pick(uint64_t key, uint64_t p, uint32_t stream, uint32_t cnt)
{
    uint64_t h = ref_splitmix64(key ^ ((p << 1) | (uint64_t)stream));
    return (uint32_t)(((h >> 32) * (uint64_t)cnt) >> 32);
}

/* ---------------------------------------------------------------------- */
/* bf16 <-> fp32 from the IEEE-754 bit layout: bf16 is the top 16 bits of  */
/* an fp32. Narrowing rounds to nearest, ties to even; NaN stays a quiet   */
/* NaN with its sign.                                                      */
/* ---------------------------------------------------------------------- */
float ref_bf16_to_f32(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

uint16_t ref_f32_to_bf16(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu) != 0)
        return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t upper = u >> 16;
    uint32_t lower = u & 0xffffu;
    if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u)))
        upper += 1; /* may carry into the exponent: correct rounding to inf */
    return (uint16_t)upper;
}

static int popcount32(uint32_t v)
{
    int c = 0;
    while (v) { c += (int)(v & 1u); v >>= 1; }
    return c;
}

/* ---------------------------------------------------------------------- */
/* Co-activation statistics (Section 3.2, Stage 1): c_ij counts the tokens */
/* that select both experts i and j, w_e the tasks of expert e. Raw counts */
/* are added into coact [E][E] for every ordered pair of distinct slots,   */
/* and into count [E] for every selection; both accumulate across calls.   */
/* ---------------------------------------------------------------------- */
int ref_coact_stats(const int32_t* topk, int64_t T, int32_t K, int32_t E,
                    uint32_t* coact, uint32_t* count)
{
    if (T < 0 || K < 1 || E < 1) return REF_EINVAL;
    for (int64_t t = 0; t < T; ++t)
        for (int32_t a = 0; a < K; ++a) {
            int32_t ea = topk[t * K + a];
            if (ea < 0 || ea >= E) return REF_EDATA;
        }
    for (int64_t t = 0; t < T; ++t) {
        const int32_t* D = topk + t * K;
        for (int32_t a = 0; a < K; ++a) {
            if (count) count[D[a]] += 1u;
            for (int32_t b = 0; b < K; ++b)
                if (a != b) coact[(int64_t)D[a] * E + D[b]] += 1u;
        }
    }
    return REF_OK;
}

/* ---------------------------------------------------------------------- */
/* Layout tables from the replica table (Section 3.1, layout {P_r};        */
/* Section 3.3, R_{e,n} and N_e).                                          */
/*   node_mask[e]     bit n set iff some rank of node n holds e  (N_e)     */
/*   rank_mask[e*N+n] bit i set iff rank n*g+i holds e           (R_{e,n}) */
/*   owner_out[e]     owner_in[e] if given, else the lowest rank holding e */
/* Rejected (REF_EDATA): an expert with no replica (coverage, Eq. 2), an   */
/* expert twice on one rank (Stage 2 placement rule), an owner that does   */
/* not hold its expert, an id outside [-1, E).                             */
/* ---------------------------------------------------------------------- */
int ref_layout_tables(int32_t N, int32_t g, int32_t E, int32_t S,
                      const int32_t* slot_table, const int32_t* owner_in,
                      uint32_t* node_mask, uint32_t* rank_mask, int32_t* owner_out)
{
    if (N < 1 || N > 16 || g < 1 || g > 32 || E < 1 || S < 1) return REF_EINVAL;
    int32_t G = N * g;
    for (int32_t e = 0; e < E; ++e) {
        node_mask[e] = 0;
        owner_out[e] = -1;
        for (int32_t n = 0; n < N; ++n) rank_mask[e * N + n] = 0;
    }
    for (int32_t r = 0; r < G; ++r) {
        int32_t n = r / g, i = r % g;
        for (int32_t s = 0; s < S; ++s) {
            int32_t e = slot_table[r * S + s];
            if (e == -1) continue;
            if (e < 0 || e >= E) return REF_EDATA;
            if (rank_mask[e * N + n] & (1u << i)) return REF_EDATA;
            rank_mask[e * N + n] |= 1u << i;
            node_mask[e] |= 1u << n;
            if (owner_out[e] < 0) owner_out[e] = r;
        }
    }
    for (int32_t e = 0; e < E; ++e) {
        if (node_mask[e] == 0) return REF_EDATA;
        if (owner_in) {
            int32_t o = owner_in[e];
            if (o < 0 || o >= G) return REF_EDATA;
            if (!(rank_mask[e * N + o / g] & (1u << (o % g)))) return REF_EDATA;
            owner_out[e] = o;
        }
    }
    return REF_OK;
}

/* RemoteMask (Section 3.3, step 1): the (N-1)-bit mask of the remote nodes
 * of a node set, where bit i stands for the i-th node other than `home`
 * in ascending id. */
static uint32_t remote_mask(uint32_t nodes, int32_t home, int32_t N)
{
    uint32_t m = 0;
    int32_t bit = 0;
    for (int32_t n = 0; n < N; ++n) {
        if (n == home) continue;
        if (nodes & (1u << n)) m |= 1u << bit;
        ++bit;
    }
    return m;
}

/* Node id of remote bit i (inverse of remote_mask's numbering). */
static int32_t remote_node(int32_t i, int32_t home)
{
    return i < home ? i : i + 1;
}

/* i-th (0-based) set bit of v, counting up from bit 0. */
static int32_t nth_set_bit(uint32_t v, uint32_t i)
{
    for (int32_t b = 0; b < 32; ++b)
        if (v & (1u << b)) {
            if (i == 0) return b;
            --i;
        }
    return -1;
}

static int32_t src_of(const int32_t* src, int64_t t, int64_t T, int32_t G)
{
    return src ? src[t] : (int32_t)(t / (T / G));
}

/* ---------------------------------------------------------------------- */
/* Communication-aware task assignment (Section 3.3, Algorithm 1).         */
/* mode 0: Algorithm 1. mode 1: every task on its expert's owner rank (the */
/* owner-only baseline that the paper compares against).                  */
/* assigned [T][K]: r_te. remote_nodes [T] (nullable): bit n set iff node  */
/* n != node(s_t) receives token t.                                        */
/* There is no load cap (Section 3.3: balance comes from the layout and    */
/* the uniform draw).                                                      */
/* ---------------------------------------------------------------------- */
int ref_assign(int32_t N, int32_t g, int32_t E,
               const uint32_t* node_mask, const uint32_t* rank_mask, const int32_t* owner,
               const int32_t* topk, const int32_t* src, int64_t T, int32_t K,
               uint64_t seed, uint64_t step, int32_t mode,
               int32_t* assigned, uint16_t* remote_nodes)
{
    int32_t G = N * g;
    if (N < 1 || N > 16 || g < 1 || g > 32 || K < 1 || K > 64 || T < 0) return REF_EINVAL;
    if (!src && T % G != 0) return REF_EINVAL;
    uint64_t key = ref_rng_key(seed, step);
    int32_t U[64];
    uint32_t m[64];
    int32_t node_of[64];

    for (int64_t t = 0; t < T; ++t) {
        const int32_t* D = topk + t * K;
        int32_t s_t = src_of(src, t, T, G);
        if (s_t < 0 || s_t >= G) return REF_EDATA;
        for (int32_t j = 0; j < K; ++j)
            if (D[j] < 0 || D[j] >= E) return REF_EDATA;
        int32_t home = s_t / g;

        if (mode == 1) {
            uint32_t nodes = 0;
            for (int32_t j = 0; j < K; ++j) {
                int32_t r = owner[D[j]];
                assigned[t * K + j] = r;
                if (r / g != home) nodes |= 1u << (r / g);
            }
            if (remote_nodes) remote_nodes[t] = (uint16_t)nodes;
            continue;
        }

        /* Step 1: select execution nodes. U_t holds the selected experts
         * with no replica on the source node; each gets its remote mask. */
        int32_t nU = 0;
        for (int32_t j = 0; j < K; ++j) {
            uint32_t Ne = node_mask[D[j]];
            if (!(Ne & (1u << home))) {
                U[nU] = j;
                m[nU] = remote_mask(Ne, home, N);
                ++nU;
            }
        }
        /* b*: the fewest remote nodes that together hold every expert of
         * U_t, a minimum cover of U_t by the nodes' expert sets; among the
         * covers of that size, the one with the smallest remote mask (the
         * order in which Algorithm 1 meets them). Node sets are tried by
         * size, and within a size by mask value, and the first cover is
         * kept. U_t empty is covered by no node at all. The set of all
         * remote nodes always covers U_t on a valid layout (every expert
         * has a replica, none of U_t's on the source node), so a cover is
         * found; the all-remote mask stands in if the layout is invalid. */
        uint32_t full = (N > 1) ? ((1u << (N - 1)) - 1u) : 0u;
        uint32_t bstar = 0;
        int found = (nU == 0);
        for (int32_t size = 1; !found && size <= N - 1; ++size) {
            for (uint32_t b = 1; !found && b <= full; ++b) {
                if (popcount32(b) != size) continue;
                int covers = 1;
                for (int32_t u = 0; u < nU; ++u)
                    if ((b & m[u]) == 0) { covers = 0; break; }
                if (covers) { bstar = b; found = 1; }
            }
        }
        if (!found) bstar = full;
        /* Each expert of U_t goes to a random node among the chosen ones
         * that hold it; the other experts stay on the source node. */
        for (int32_t j = 0; j < K; ++j) node_of[j] = home;
        for (int32_t u = 0; u < nU; ++u) {
            uint32_t cand = bstar & m[u];
            int64_t p = t * K + U[u];
            uint32_t k = ref_pick(key, (uint64_t)p, 0, (uint32_t)popcount32(cand));
            node_of[U[u]] = remote_node(nth_set_bit(cand, k), home);
        }
        /* Step 2: select execution ranks uniformly among the node's ranks
         * that hold the expert. */
        for (int32_t j = 0; j < K; ++j) {
            int32_t n = node_of[j];
            uint32_t R = rank_mask[D[j] * N + n];
            int64_t p = t * K + j;
            uint32_t k = ref_pick(key, (uint64_t)p, 1, (uint32_t)popcount32(R));
            assigned[p] = n * g + nth_set_bit(R, k);
        }
        if (remote_nodes) {
            uint32_t nodes = 0;
            for (int32_t i = 0; i < N - 1; ++i)
                if (bstar & (1u << i)) nodes |= 1u << remote_node(i, home);
            remote_nodes[t] = (uint16_t)nodes;
        }
    }
    return REF_OK;
}

/* ---------------------------------------------------------------------- */
/* Dispatch layout (the EP dispatch of Section 1 / Fig. 1, one row per    */
/* (token, expert) pair). Bucket of pair p = (s_t, r_p), buckets in        */
/* row-major order; each bucket keeps pairs in increasing p.               */
/*   counts [G][G]      pairs per (source, destination)                    */
/*   offsets [G*G+1]    exclusive prefix sum of counts, offsets[G*G]=total */
/*   pos [T][K]         row of pair p in the packed buffer                 */
/*   packed [T*K][d]    packed[pos[p]] = x[t] (bf16 bits), nullable        */
/* ---------------------------------------------------------------------- */
int ref_dispatch(const int32_t* assigned, const int32_t* src, int64_t T, int32_t K, int32_t G,
                 const uint16_t* x, int64_t d,
                 int32_t* counts, int64_t* offsets, int32_t* pos, uint16_t* packed)
{
    if (T < 0 || K < 1 || G < 1 || d < 0) return REF_EINVAL;
    if (!src && T % G != 0) return REF_EINVAL;
    int64_t GG = (int64_t)G * G;
    for (int64_t b = 0; b < GG; ++b) counts[b] = 0;
    for (int64_t t = 0; t < T; ++t) {
        int32_t s = src_of(src, t, T, G);
        if (s < 0 || s >= G) return REF_EDATA;
        for (int32_t j = 0; j < K; ++j) {
            int32_t r = assigned[t * K + j];
            if (r < 0 || r >= G) return REF_EDATA;
            counts[(int64_t)s * G + r] += 1;
        }
    }
    int64_t run = 0;
    for (int64_t b = 0; b < GG; ++b) {
        offsets[b] = run;
        run += counts[b];
    }
    offsets[GG] = run;
    int64_t* cursor = (int64_t*)malloc((size_t)(GG > 0 ? GG : 1) * sizeof(int64_t));
    if (!cursor) return REF_EINVAL;
    for (int64_t b = 0; b < GG; ++b) cursor[b] = offsets[b];
    for (int64_t t = 0; t < T; ++t) {
        int32_t s = src_of(src, t, T, G);
        for (int32_t j = 0; j < K; ++j) {
            int64_t p = t * K + j;
            int64_t b = (int64_t)s * G + assigned[p];
            int64_t row = cursor[b]++;
            pos[p] = (int32_t)row;
            if (packed)
                for (int64_t c = 0; c < d; ++c) packed[row * d + c] = x[t * d + c];
        }
    }
    free(cursor);
    return REF_OK;
}

/* ---------------------------------------------------------------------- */
/* Node-deduplicated dispatch layout (Section 1 and Section 3.1: a token  */
/* crosses to a node once, however many ranks there need it, and is then  */
/* forwarded inside that node). Token t has one row per distinct node     */
/*   n in { node(r_tj) : j = 0..K-1 },                                    */
/* its own node included, so the rows whose node differs from node(s_t)   */
/* number exactly the V of Eq. 1. Bucket of row (t, n) = (s_t, n), in      */
/* row-major order over [G][N]; a bucket keeps its rows in increasing t.   */
/*   counts [G][N]      rows per (source rank, destination node)           */
/*   offsets [G*N+1]    exclusive prefix sum of counts, offsets[G*N]=total */
/*   node_pos [T][N]    row of (t, n), or -1 if no slot of t goes to n     */
/*   fwd [rows]         forwarding mask of the row: bit i set iff some     */
/*                      slot of its token is assigned to rank n*g + i      */
/*   row_token [rows]   t of the row (nullable)                            */
/*   packed [rows][d]   packed[row] = x[t] (bf16 bits), nullable           */
/* rows <= T * min(K, N).                                                  */
/* ---------------------------------------------------------------------- */
int ref_node_dispatch(const int32_t* assigned, const int32_t* src, int64_t T, int32_t K,
                      int32_t N, int32_t g, const uint16_t* x, int64_t d,
                      int32_t* counts, int64_t* offsets, int32_t* node_pos, uint32_t* fwd,
                      int32_t* row_token, uint16_t* packed)
{
    if (T < 0 || K < 1 || N < 1 || N > 32 || g < 1 || g > 32 || d < 0) return REF_EINVAL;
    int32_t G = N * g;
    if (!src && T % G != 0) return REF_EINVAL;
    int64_t GN = (int64_t)G * N;
    uint32_t* mask = (uint32_t*)malloc((size_t)N * sizeof(uint32_t));
    int64_t* cursor = (int64_t*)malloc((size_t)(GN > 0 ? GN : 1) * sizeof(int64_t));
    if (!mask || !cursor) {
        free(mask);
        free(cursor);
        return REF_EINVAL;
    }
    int rc = REF_OK;
    for (int64_t b = 0; b < GN; ++b) counts[b] = 0;
    /* pass 1: which nodes each token reaches */
    for (int64_t t = 0; t < T && rc == REF_OK; ++t) {
        int32_t s = src_of(src, t, T, G);
        if (s < 0 || s >= G) rc = REF_EDATA;
        for (int32_t n = 0; n < N; ++n) mask[n] = 0;
        for (int32_t j = 0; j < K && rc == REF_OK; ++j) {
            int32_t r = assigned[t * K + j];
            if (r < 0 || r >= G) rc = REF_EDATA;
            else mask[r / g] |= 1u << (r % g);
        }
        for (int32_t n = 0; n < N && rc == REF_OK; ++n)
            if (mask[n]) counts[(int64_t)s * N + n] += 1;
    }
    if (rc == REF_OK) {
        int64_t run = 0;
        for (int64_t b = 0; b < GN; ++b) {
            offsets[b] = run;
            run += counts[b];
        }
        offsets[GN] = run;
        for (int64_t b = 0; b < GN; ++b) cursor[b] = offsets[b];
        /* pass 2: rows in increasing t within each bucket */
        for (int64_t t = 0; t < T; ++t) {
            int32_t s = src_of(src, t, T, G);
            for (int32_t n = 0; n < N; ++n) mask[n] = 0;
            for (int32_t j = 0; j < K; ++j) {
                int32_t r = assigned[t * K + j];
                mask[r / g] |= 1u << (r % g);
            }
            for (int32_t n = 0; n < N; ++n) {
                if (!mask[n]) {
                    node_pos[t * N + n] = -1;
                    continue;
                }
                int64_t row = cursor[(int64_t)s * N + n]++;
                node_pos[t * N + n] = (int32_t)row;
                fwd[row] = mask[n];
                if (row_token) row_token[row] = (int32_t)t;
                if (packed)
                    for (int64_t c = 0; c < d; ++c) packed[row * d + c] = x[t * d + c];
            }
        }
    }
    free(mask);
    free(cursor);
    return rc;
}

/* ---------------------------------------------------------------------- */
/* Combine and weighted sum (Fig. 1, last stage): token t gets            */
/*   y[t][c] = bf16( sum_j gates[t][j] * expert_out[pos[t][j]][c] )       */
/* accumulated in fp32 from 0, one fused multiply-add per slot, j = 0..K-1.*/
/* y32 (nullable) receives the fp32 sums. Rows outside [0, rows) add 0.    */
/* ---------------------------------------------------------------------- */
int ref_combine(const uint16_t* expert_out, int64_t rows, const int32_t* pos, const float* gates,
                int64_t T, int32_t K, int64_t d, uint16_t* y, float* y32)
{
    if (T < 0 || K < 1 || d < 0) return REF_EINVAL;
    for (int64_t t = 0; t < T; ++t)
        for (int64_t c = 0; c < d; ++c) {
            float acc = 0.0f;
            for (int32_t j = 0; j < K; ++j) {
                int64_t row = pos[t * K + j];
                if (row < 0 || row >= rows) continue;
                acc = fmaf(gates[t * K + j], ref_bf16_to_f32(expert_out[row * d + c]), acc);
            }
            if (y) y[t * d + c] = ref_f32_to_bf16(acc);
            if (y32) y32[t * d + c] = acc;
        }
    return REF_OK;
}

/* ---------------------------------------------------------------------- */
/* Node-level combine, the reverse of the node-deduplicated dispatch      */
/* (Section 1 and Section 3.1: a token's results leave a node once). On    */
/* node n the slots of token t whose rank r_tj lies on n (r_tj / g = n)   */
/* are summed first, fp32 from 0, one fused multiply-add per slot in slot */
/* order, and the partial is rounded to bf16:                             */
/*   part[t][n][c] = bf16( sum_{j on n} gates[t][j] * eo[pos[t][j]][c] )  */
/* It is stored in row node_pos[t][n] of partial, the row the dispatch     */
/* used for (t, n). At the source the partials are summed, fp32 from 0,    */
/* in increasing n, and rounded once more:                                */
/*   y[t][c] = bf16( sum_{n : node_pos[t][n] valid} float(part[t][n][c]) ) */
/* Skipped: slots with a rank outside [0, N*g) or a row outside [0, rows); */
/* node rows outside [0, node_rows) (neither written nor summed). A valid  */
/* node row with no slot of its token on the node holds zero.             */
/* ---------------------------------------------------------------------- */
int ref_node_combine(const uint16_t* expert_out, int64_t rows, const int32_t* pos,
                     const int32_t* assigned, const float* gates, const int32_t* node_pos,
                     int64_t T, int32_t K, int32_t N, int32_t g, int64_t d, int64_t node_rows,
                     uint16_t* partial, uint16_t* y)
{
    if (T < 0 || K < 1 || N < 1 || N > 32 || g < 1 || g > 32 || d < 0 || node_rows < 0)
        return REF_EINVAL;
    int32_t G = N * g;
    /* node side: one partial row per (token, node) */
    for (int64_t t = 0; t < T; ++t)
        for (int32_t n = 0; n < N; ++n) {
            int64_t nrow = node_pos[t * N + n];
            if (nrow < 0 || nrow >= node_rows) continue;
            for (int64_t c = 0; c < d; ++c) {
                float acc = 0.0f;
                for (int32_t j = 0; j < K; ++j) {
                    int32_t r = assigned[t * K + j];
                    int64_t row = pos[t * K + j];
                    if (r < 0 || r >= G || r / g != n) continue;
                    if (row < 0 || row >= rows) continue;
                    acc = fmaf(gates[t * K + j], ref_bf16_to_f32(expert_out[row * d + c]), acc);
                }
                partial[nrow * d + c] = ref_f32_to_bf16(acc);
            }
        }
    /* source side: the partials of each token, in increasing n */
    for (int64_t t = 0; t < T; ++t)
        for (int64_t c = 0; c < d; ++c) {
            float acc = 0.0f;
            for (int32_t n = 0; n < N; ++n) {
                int64_t nrow = node_pos[t * N + n];
                if (nrow < 0 || nrow >= node_rows) continue;
                acc = acc + ref_bf16_to_f32(partial[nrow * d + c]);
            }
            y[t * d + c] = ref_f32_to_bf16(acc);
        }
    return REF_OK;
}

/* ---------------------------------------------------------------------- */
/* Traffic model (Eq. 1) and load: V = sum over tokens of the number of    */
/* distinct nodes other than node(s_t) among the token's assigned ranks;   */
/* cross_pairs counts pairs whose rank is on another node; load[r] counts  */
/* pairs assigned to rank r (w summed over the rank's replicas).           */
/* ---------------------------------------------------------------------- */
int ref_traffic(const int32_t* assigned, const int32_t* src, int64_t T, int32_t K,
                int32_t N, int32_t g, int64_t* V, int64_t* cross_pairs, int64_t* load)
{
    int32_t G = N * g;
    if (!src && T % G != 0) return REF_EINVAL;
    *V = 0;
    *cross_pairs = 0;
    for (int32_t r = 0; r < G; ++r) load[r] = 0;
    for (int64_t t = 0; t < T; ++t) {
        int32_t home = src_of(src, t, T, G) / g;
        uint32_t nodes = 0;
        for (int32_t j = 0; j < K; ++j) {
            int32_t r = assigned[t * K + j];
            if (r < 0 || r >= G) return REF_EDATA;
            load[r] += 1;
            if (r / g != home) {
                nodes |= 1u << (r / g);
                *cross_pairs += 1;
            }
        }
        *V += popcount32(nodes);
    }
    return REF_OK;
}

/* ---------------------------------------------------------------------- */
/* Exponential moving averages of the planner's statistics (Section 3.2:  */
/* Stage 1 keeps EMAs of w_e, the tasks of expert e, and of c_ij, the      */
/* tokens selecting both i and j; Stage 2 keeps an EMA of each replica's   */
/* tasks). The decay is not given in the paper; it is a parameter here.    */
/* One update of an EMA m with this step's count x, in fp32:              */
/*   init:      m = x                                                      */
/*   otherwise: m = fma(decay, m, (1 - decay) * x)                         */
/* where x is the count converted to fp32 and 1 - decay is rounded to      */
/* fp32 once. clear: the counts are set to 0 after they are read.          */
/* ---------------------------------------------------------------------- */
int ref_count_ema(uint32_t* counts, int64_t n, float decay, int32_t init, int32_t clear,
                  float* ema)
{
    if (n < 0 || !(decay >= 0.0f && decay <= 1.0f)) return REF_EINVAL;
    float gain = 1.0f - decay;
    for (int64_t i = 0; i < n; ++i) {
        float x = (float)counts[i];
        if (init) ema[i] = x;
        else ema[i] = fmaf(decay, ema[i], gain * x);
        if (clear) counts[i] = 0;
    }
    return REF_OK;
}

/* ---------------------------------------------------------------------- */
/* Ochiai similarity of experts i and j (Section 1, footnote on Fig. 3):  */
/* with A_i the set of tokens that select expert i,                        */
/*   O_ij = |A_i & A_j| / sqrt(|A_i| |A_j|),                               */
/* from the co-activation counts: |A_i & A_j| = coact[i][j] for i != j and */
/* |A_i| = count[i]. O_ii = 1 for an expert some token selects. A pair     */
/* with no common token, or an expert no token selects, gives 0. In fp32: */
/*   O_ij = (float)c / sqrtf((float)n_i * (float)n_j).                     */
/* ---------------------------------------------------------------------- */
int ref_ochiai(const uint32_t* coact, const uint32_t* count, int32_t E, float* ochiai)
{
    if (E < 1) return REF_EINVAL;
    for (int32_t i = 0; i < E; ++i)
        for (int32_t j = 0; j < E; ++j) {
            uint32_t c = i == j ? count[i] : coact[(int64_t)i * E + j];
            float o = 0.0f;
            if (c != 0 && count[i] != 0 && count[j] != 0)
                o = (float)c / sqrtf((float)count[i] * (float)count[j]);
            ochiai[(int64_t)i * E + j] = o;
        }
    return REF_OK;
}

/* ---------------------------------------------------------------------- */
/* Per-replica workload (Section 3.1: w_er, the tasks of expert e executed */
/* by its replica on rank r). load [E][G] += counts; pairs with an id or   */
/* rank out of range are skipped.                                          */
/* ---------------------------------------------------------------------- */
int ref_replica_load(const int32_t* topk, const int32_t* assigned, int64_t T, int32_t K,
                     int32_t E, int32_t G, uint32_t* load)
{
    if (T < 0 || K < 1 || E < 1 || G < 1) return REF_EINVAL;
    for (int64_t p = 0; p < T * K; ++p) {
        int32_t e = topk[p], r = assigned[p];
        if (e < 0 || e >= E || r < 0 || r >= G) continue;
        load[(int64_t)e * G + r] += 1u;
    }
    return REF_OK;
}

/* ---------------------------------------------------------------------- */
/* Per-step intra-node rebalancing (Section 3.2, Stage 2): for each node,  */
/* sort the node's replicas by estimated workload, heaviest first (ties:   */
/* smaller expert id, then smaller previous rank), and give each in turn to */
/* the least-loaded rank of the node (ties: smaller rank) that has a free  */
/* slot and holds no replica of the same expert. A node where some replica */
/* finds no such rank keeps its previous placement. rank_load receives the */
/* fp32 sums of each rank's replica loads in placement order.              */
/* ---------------------------------------------------------------------- */
struct ref_rep { float load; int32_t e, r; };

static int rep_before(const struct ref_rep* a, const struct ref_rep* b)
{
    if (a->load != b->load) return a->load > b->load;
    if (a->e != b->e) return a->e < b->e;
    return a->r < b->r;
}

int ref_intra_node_rebalance(int32_t N, int32_t g, int32_t E, int32_t S,
                             const int32_t* slot, const int32_t* owner_in, const float* rload,
                             int32_t* new_slot, int32_t* new_owner, float* rank_load)
{
    int32_t G = N * g;
    if (N < 1 || g < 1 || E < 1 || S < 1) return REF_EINVAL;
    uint32_t* node_mask = (uint32_t*)calloc((size_t)E, sizeof(uint32_t));
    uint32_t* rank_mask = (uint32_t*)calloc((size_t)E * N, sizeof(uint32_t));
    int32_t* owner = (int32_t*)calloc((size_t)E, sizeof(int32_t));
    struct ref_rep* reps = (struct ref_rep*)malloc((size_t)g * S * sizeof(struct ref_rep));
    int32_t* dest = (int32_t*)malloc((size_t)g * S * sizeof(int32_t));
    float* load = (float*)malloc((size_t)g * sizeof(float));
    int32_t* used = (int32_t*)malloc((size_t)g * sizeof(int32_t));
    int rc = REF_OK;
    if (!node_mask || !rank_mask || !owner || !reps || !dest || !load || !used) {
        rc = REF_EINVAL;
        goto done;
    }
    rc = ref_layout_tables(N, g, E, S, slot, owner_in, node_mask, rank_mask, owner);
    if (rc != REF_OK) goto done;
    for (int32_t r = 0; r < G; ++r)
        for (int32_t k = 0; k < S; ++k) {
            int32_t e = slot[r * S + k];
            if (e < 0) continue;
            float l = rload[(int64_t)e * G + r];
            if (!(l >= 0.0f) || isinf(l)) { rc = REF_EDATA; goto done; }
        }
    for (int32_t e = 0; e < E; ++e) new_owner[e] = owner[e];
    for (int32_t n = 0; n < N; ++n) {
        int32_t nrep = 0;
        for (int32_t i = 0; i < g; ++i)
            for (int32_t k = 0; k < S; ++k) {
                int32_t r = n * g + i, e = slot[r * S + k];
                if (e < 0) continue;
                reps[nrep].load = rload[(int64_t)e * G + r];
                reps[nrep].e = e;
                reps[nrep].r = r;
                ++nrep;
            }
        /* insertion sort, heaviest first */
        for (int32_t a = 1; a < nrep; ++a) {
            struct ref_rep x = reps[a];
            int32_t b = a - 1;
            while (b >= 0 && rep_before(&x, &reps[b])) { reps[b + 1] = reps[b]; --b; }
            reps[b + 1] = x;
        }
        for (int32_t i = 0; i < g; ++i) { load[i] = 0.0f; used[i] = 0; }
        int placed_all = 1;
        for (int32_t q = 0; q < nrep && placed_all; ++q) {
            int32_t best = -1;
            for (int32_t i = 0; i < g; ++i) {
                int holds = 0;
                for (int32_t u = 0; u < q; ++u)
                    if (dest[u] == i && reps[u].e == reps[q].e) holds = 1;
                if (used[i] >= S || holds) continue;
                if (best < 0 || load[i] < load[best]) best = i;
            }
            if (best < 0) { placed_all = 0; break; }
            dest[q] = best;
            load[best] += reps[q].load;
            used[best] += 1;
        }
        if (placed_all) {
            for (int32_t i = 0; i < g; ++i) {
                int32_t r = n * g + i, k = 0;
                for (int32_t q = 0; q < nrep; ++q)
                    if (dest[q] == i) new_slot[r * S + k++] = reps[q].e;
                for (; k < S; ++k) new_slot[r * S + k] = -1;
                if (rank_load) rank_load[r] = load[i];
            }
            for (int32_t q = 0; q < nrep; ++q)
                if (owner[reps[q].e] == reps[q].r) new_owner[reps[q].e] = n * g + dest[q];
        } else {
            for (int32_t i = 0; i < g; ++i) {
                int32_t r = n * g + i;
                float l = 0.0f;
                for (int32_t k = 0; k < S; ++k) {
                    int32_t e = slot[r * S + k];
                    new_slot[r * S + k] = e;
                    if (e >= 0) l += rload[(int64_t)e * G + r];
                }
                if (rank_load) rank_load[r] = l;
            }
        }
    }
done:
    free(node_mask); free(rank_mask); free(owner); free(reps); free(dest); free(load); free(used);
    return rc;
}

/* ---------------------------------------------------------------------- */
/* Periodic global planning (Section 3.2, Stage 1; Eq. 3 and its MILP in   */
/* the appendix). The paper solves Eq. 3 exactly with a MILP solver; this  */
/* is a greedy heuristic for the same objective and constraints, stated    */
/* step by step below, and this oracle follows those steps literally.      */
/*                                                                        */
/* Objective: sum over nodes n and pairs i < j of c_ij [i, j both on n].   */
/* Constraints: every expert on some rank; at most S replicas per rank; no */
/* expert twice on a rank; planned work l_er >= 0 only where e is held,    */
/* sum_r l_er = w_e; sum_e l_er <= cap = (1 + eps) W / G per rank, where   */
/* W = sum_e w_e. Pair weights are quantised to q_ij = llrint(256 c_ij) in */
/* int64 so that every gain is an exact integer sum.                       */
/*                                                                        */
/* gain(e, n) = sum of q_ex over experts x != e already on node n.         */
/* need(x)    = 1 if x <= cap, else ceil(x / cap): ranks a share x needs.  */
/*                                                                        */
/* 1. Work placement. Experts in decreasing w (ties: smaller id). Each    */
/*    takes nodes one at a time until its work is placed: among nodes not */
/*    holding it with a free slot, the best by (the whole remainder fits  */
/*    in the node's spare work g cap - work and its free slots, some      */
/*    spare work left, spare work, gain), ties to the smaller node. A     */
/*    fitting node takes the remainder; otherwise the node takes what its */
/*    spare work and free slots allow (if nothing, the remainder). The    */
/*    share reserves need(share) slots of the node, at most its free      */
/*    slots and g. If every node was tried, the rest goes to the last one.*/
/*    Steps 1 and 1b use g S - R slots per node, R = min(g, (G S - sum_e  */
/*    need(w_e)) / N) (integer division, 0 if negative): the free slots   */
/*    the repair of step 2 may split work into. Step 1 picks among nodes  */
/*    within g S - R slots first, and uses all g S slots when that finds  */
/*    no node at all, or only non-fitting ones while a node fits with    */
/*    all slots.                                                          */
/*    Local search: an expert placed whole on one node in one slot is     */
/*    single. Sweeps over single experts a in increasing id apply, for    */
/*    each a, the best of (ties: moves before swaps, then smaller node or */
/*    smaller b)                                                          */
/*      move a to node m with a free slot:                                */
/*        delta = gain(a, m) - gain(a, n_a)                               */
/*      swap a with a single b on another node:                           */
/*        delta = gain(a, n_b) - gain(a, n_a) + gain(b, n_a)              */
/*                - gain(b, n_b) - 2 q_ab                                 */
/*    if its delta is positive and every node it changes ends with work   */
/*    at most g cap or no more than before. Sweeps repeat until one       */
/*    changes nothing (at most 64 sweeps).                                */
/* 2. Ranks, node by node. Each share is cut into need(share) equal      */
/*    pieces; pieces in decreasing work (ties: smaller e, earlier piece)  */
/*    go to the rank of the node with least planned work (ties: fewer     */
/*    replicas, smaller rank) that holds fewer than min(S, ceil(pieces /  */
/*    g)) replicas, so that free slots stay spread over the ranks,        */
/*    and does not hold the expert. If some piece finds none, the node is */
/*    laid out round-robin instead: experts by decreasing piece count     */
/*    (ties: smaller e), the                                              */
/*    node's p-th piece on rank p mod g.                                  */
/*    Repair, an augmenting-path step on the flow network expert -> rank: */
/*    while the most loaded rank h of the node (ties: smaller) exceeds    */
/*    cap, search breadth-first from h: from rank a, for each expert e    */
/*    with work on a (increasing e), each unvisited rank b of the node    */
/*    (increasing) that holds e, or has a free slot, is reached through   */
/*    e. The first reached rank t below cap ends the search; the work     */
/*    min(load_h - cap, cap - load_t, the work of each path expert on its */
/*    rank) moves along the path, adding replicas where b did not hold e. */
/*    If no such rank is reachable and h has a free slot, a slot swap:    */
/*    eh is the expert with the most work on h (ties: smaller e); among   */
/*    the under-cap ranks u with no free slot and without eh, the least   */
/*    loaded (ties: smaller) that holds an expert x with less work than   */
/*    eh has on h and not held by h, x the one with least work (ties:     */
/*    smaller). x moves whole from u to h, then m = min(load_h - cap +    */
/*    w_x, cap - load_u + w_x, l_eh,h) of eh moves to a new replica on u, */
/*    if m > w_x. Stop when neither applies or a path move is below       */
/*    cap 1e-12 (at most 4 g^2 S moves).                                  */
/* 2b. Global repair. While the most loaded rank h of all (ties: smaller) */
/*    exceeds cap, the same breadth-first search over the ranks of all    */
/*    nodes (increasing id), so that a node left above its ranks' caps    */
/*    can pass work to another node. It searches first through ranks that */
/*    already hold the path's expert, and only when that reaches no       */
/*    target also through free slots (a new replica, which makes its     */
/*    expert a member of that node). A target has room above cap 1e-12:   */
/*    cap - load_t > cap 1e-12. It stops when no rank exceeds cap, no     */
/*    target is reachable, or a move is below cap 1e-12 (at most 4 G S   */
/*    moves).                                                             */
/* 3. Co-activation replicas. While some (e, n) with e not on n, a free   */
/*    slot on n and positive gain exists: add the one with the largest    */
/*    gain (ties: larger w, smaller e, smaller n) on the rank of n with   */
/*    fewest replicas (ties: smaller), with no planned work.              */
/* Retries. If the plan exceeds the cap, steps 1 to 3 run again with the */
/* node work bound of step 1 and its local search lowered to f g cap,     */
/* f = 0.98, 0.95, 0.90 in turn, which leaves work slack on every node    */
/* for steps 2 and 2b. The first plan within the cap is returned; if none */
/* is (or a retry finds no slot for some expert), the plan with f = 1.    */
/* owner[e]: the rank with the most planned work for e (ties: smaller).   */
/* plan [E][G]: planned work l_er (fp32 of the double sums); objective:    */
/* the quantised objective / 256; feasible: every rank's planned work is   */
/* at most cap (1 + 1e-9).                                                */
/* ---------------------------------------------------------------------- */
static int64_t plan_q(const int64_t* q, int32_t E, int32_t a, int32_t b)
{
    if (a == b) return 0;
    return a < b ? q[(int64_t)a * E + b] : q[(int64_t)b * E + a];
}

static int64_t plan_gain(const int64_t* q, const uint8_t* on, int32_t E, int32_t N, int32_t e,
                         int32_t n)
{
    int64_t s = 0;
    for (int32_t x = 0; x < E; ++x)
        if (x != e && on[(int64_t)x * N + n]) s += plan_q(q, E, e, x);
    return s;
}

static int64_t plan_need(double x, double cap)
{
    if (x <= cap) return 1;
    return (int64_t)ceil(x / cap);
}

struct plan_piece { double load; int32_t e, c; };

static int piece_before(const struct plan_piece* a, const struct plan_piece* b)
{
    if (a->load != b->load) return a->load > b->load;
    if (a->e != b->e) return a->e < b->e;
    return a->c < b->c;
}

/* replicas on rank r: slots in use */
static int32_t plan_used(const int32_t* slot_table, int32_t S, int32_t r)
{
    int32_t k = 0;
    while (k < S && slot_table[(int64_t)r * S + k] >= 0) ++k;
    return k;
}

static int plan_holds(const int32_t* slot_table, int32_t S, int32_t r, int32_t e)
{
    for (int32_t k = 0; k < S; ++k)
        if (slot_table[(int64_t)r * S + k] == e) return 1;
    return 0;
}

static double plan_rank_load(const double* pl, int32_t E, int32_t G, int32_t r)
{
    double l = 0.0;
    for (int32_t e = 0; e < E; ++e) l += pl[(int64_t)e * G + r];
    return l;
}

static int plan_once(int32_t N, int32_t g, int32_t E, int32_t S, const float* coact_ema,
                     const float* count_ema, float eps, double node_frac, int32_t* slot_table,
                     int32_t* owner, float* plan, double* objective, int32_t* feasible)
{
    if (N < 1 || N > 16 || g < 1 || g > 32 || E < 1 || E > 4096 || S < 1) return REF_EINVAL;
    if (!(eps >= 0.0f) || isinf(eps)) return REF_EINVAL;
    int32_t G = N * g;
    if ((int64_t)G * S < E) return REF_EINVAL;
    for (int32_t e = 0; e < E; ++e)
        if (!(count_ema[e] >= 0.0f) || isinf(count_ema[e])) return REF_EDATA;
    for (int32_t i = 0; i < E; ++i)
        for (int32_t j = i + 1; j < E; ++j) {
            float c = coact_ema[(int64_t)i * E + j];
            /* q <= 2^36: the objective, at most 16 nodes x E(E-1)/2 < 2^23 */
            /* pairs of them, stays below 2^63 */
            if (!(c >= 0.0f) || !(c <= 268435456.0f)) return REF_EDATA; /* 2^28 */
        }

    int rc = REF_OK;
    int64_t* q = (int64_t*)calloc((size_t)E * E, sizeof(int64_t));
    uint8_t* on = (uint8_t*)calloc((size_t)E * N, 1);
    double* share = (double*)calloc((size_t)E * N, sizeof(double));
    int64_t* pieces = (int64_t*)calloc((size_t)E * N, sizeof(int64_t));
    int32_t* order = (int32_t*)malloc((size_t)E * sizeof(int32_t));
    int64_t* used = (int64_t*)calloc((size_t)N, sizeof(int64_t));
    double* work = (double*)calloc((size_t)N, sizeof(double));
    double* pl = (double*)calloc((size_t)E * G, sizeof(double));
    struct plan_piece* items = (struct plan_piece*)malloc((size_t)g * S * sizeof(struct plan_piece));
    double* rload = (double*)calloc((size_t)g, sizeof(double));
    int32_t* dest = (int32_t*)malloc((size_t)g * S * sizeof(int32_t));
    if (!q || !on || !share || !pieces || !order || !used || !work || !pl || !items || !rload ||
        !dest) {
        rc = REF_EINVAL;
        goto done;
    }
    for (int32_t i = 0; i < E; ++i)
        for (int32_t j = i + 1; j < E; ++j)
            q[(int64_t)i * E + j] = (int64_t)llrint(256.0 * (double)coact_ema[(int64_t)i * E + j]);
    for (int64_t i = 0; i < (int64_t)G * S; ++i) slot_table[i] = -1;

    double W = 0.0;
    for (int32_t e = 0; e < E; ++e) W += (double)count_ema[e];
    double cap = (1.0 + (double)eps) * W / (double)G;
    double node_cap = (double)g * cap * node_frac;
    int64_t all_slots = (int64_t)g * S;
    /* slots each node keeps free through step 1 for the repair of step 2 */
    int64_t total_need = 0;
    for (int32_t e = 0; e < E; ++e) total_need += plan_need((double)count_ema[e], cap);
    int64_t reserve = (int64_t)G * S > total_need ? ((int64_t)G * S - total_need) / N : 0;
    if (reserve > g) reserve = g;
    int64_t node_slots = all_slots - reserve;

    /* experts by decreasing w, ties to the smaller id (insertion sort) */
    for (int32_t e = 0; e < E; ++e) {
        int32_t k = e;
        while (k > 0 && count_ema[order[k - 1]] < count_ema[e]) {
            order[k] = order[k - 1];
            --k;
        }
        order[k] = e;
    }

    /* 1. work placement */
    for (int32_t oi = 0; oi < E; ++oi) {
        int32_t e = order[oi];
        double rem = (double)count_ema[e];
        int placed = 0, last = -1;
        while (!placed || rem > 0.0) {
            /* candidates with the repair reserve kept; a fitting node that
               needs the reserved slots beats a non-fitting one */
            int32_t best = -1, bfits = 0, broom = 0;
            int64_t bgain = 0;
            double bspare = 0.0;
            int64_t slots_now = node_slots;
            for (int32_t pass = 0; pass < 2; ++pass) {
                int64_t lim_slots = pass == 0 ? node_slots : all_slots;
                int32_t pb = -1, pfits = 0, proom = 0;
                int64_t pgain = 0;
                double pspare = 0.0;
                for (int32_t n = 0; n < N; ++n) {
                    if (on[(int64_t)e * N + n] || used[n] >= lim_slots) continue;
                    int64_t nfree = lim_slots - used[n];
                    int64_t lim = nfree < g ? nfree : g;
                    double spare = node_cap - work[n];
                    int fits = rem <= spare && plan_need(rem, cap) <= lim;
                    int room = spare > 0.0;
                    int64_t gn = plan_gain(q, on, E, N, e, n);
                    int better = pb < 0 || fits > pfits ||
                                 (fits == pfits && (room > proom ||
                                  (room == proom && (spare > pspare ||
                                   (spare == pspare && gn > pgain)))));
                    if (better) {
                        pb = n;
                        pfits = fits;
                        proom = room;
                        pgain = gn;
                        pspare = spare;
                    }
                }
                if (pb >= 0 && (best < 0 || (pfits && !bfits))) {
                    best = pb;
                    bfits = pfits;
                    broom = proom;
                    bgain = pgain;
                    bspare = pspare;
                    slots_now = lim_slots;
                }
                if (best >= 0 && bfits) break;
            }
            (void)broom;
            (void)bgain;
            if (best < 0) {
                if (!placed) {
                    rc = REF_EDATA; /* no free slot left for this expert */
                    goto done;
                }
                share[(int64_t)e * N + last] += rem; /* every node tried */
                work[last] += rem;
                rem = 0.0;
                break;
            }
            int64_t nfree = slots_now - used[best];
            int64_t lim = nfree < g ? nfree : g;
            double take = rem;
            if (!bfits) {
                if (bspare < take) take = bspare;
                if ((double)lim * cap < take) take = (double)lim * cap;
                if (!(take > 0.0)) take = rem;
            }
            int64_t kk = plan_need(take, cap);
            if (kk > lim) kk = lim;
            on[(int64_t)e * N + best] = 1;
            share[(int64_t)e * N + best] = take;
            pieces[(int64_t)e * N + best] = kk;
            used[best] += kk;
            work[best] += take;
            rem -= take;
            placed = 1;
            last = best;
        }
    }

    /* 1b. local search over single experts */
    for (int32_t sweep = 0; sweep < 64; ++sweep) {
        int changed = 0;
        for (int32_t a = 0; a < E; ++a) {
            int32_t na = -1, cnt = 0;
            for (int32_t n = 0; n < N; ++n)
                if (on[(int64_t)a * N + n]) {
                    na = n;
                    ++cnt;
                }
            if (cnt != 1 || pieces[(int64_t)a * N + na] != 1) continue;
            double wa = (double)count_ema[a];
            int64_t ga = plan_gain(q, on, E, N, a, na);
            int64_t bd = 0;
            int32_t bm = -1, bb = -1;
            for (int32_t m = 0; m < N; ++m) {
                if (m == na || used[m] >= node_slots) continue;
                double nw = work[m] + wa;
                if (!(nw <= node_cap || nw <= work[m])) continue;
                int64_t dl = plan_gain(q, on, E, N, a, m) - ga;
                if (dl > bd) {
                    bd = dl;
                    bm = m;
                }
            }
            for (int32_t b = 0; b < E; ++b) {
                if (b == a) continue;
                int32_t nb = -1, cb = 0;
                for (int32_t n = 0; n < N; ++n)
                    if (on[(int64_t)b * N + n]) {
                        nb = n;
                        ++cb;
                    }
                if (cb != 1 || pieces[(int64_t)b * N + nb] != 1 || nb == na) continue;
                double wb = (double)count_ema[b];
                double wna = work[na] - wa + wb, wnb = work[nb] - wb + wa;
                if (!(wna <= node_cap || wna <= work[na])) continue;
                if (!(wnb <= node_cap || wnb <= work[nb])) continue;
                int64_t dl = plan_gain(q, on, E, N, a, nb) - ga + plan_gain(q, on, E, N, b, na) -
                             plan_gain(q, on, E, N, b, nb) - 2 * plan_q(q, E, a, b);
                if (dl > bd) {
                    bd = dl;
                    bm = -1;
                    bb = b;
                }
            }
            if (bm >= 0) {
                on[(int64_t)a * N + na] = 0;
                on[(int64_t)a * N + bm] = 1;
                share[(int64_t)a * N + bm] = share[(int64_t)a * N + na];
                share[(int64_t)a * N + na] = 0.0;
                pieces[(int64_t)a * N + bm] = 1;
                pieces[(int64_t)a * N + na] = 0;
                used[na] -= 1;
                used[bm] += 1;
                work[na] = work[na] - wa;
                work[bm] = work[bm] + wa;
                changed = 1;
            } else if (bb >= 0) {
                int32_t nb = -1;
                for (int32_t n = 0; n < N; ++n)
                    if (on[(int64_t)bb * N + n]) nb = n;
                double wb = (double)count_ema[bb];
                on[(int64_t)a * N + na] = 0;
                on[(int64_t)a * N + nb] = 1;
                on[(int64_t)bb * N + nb] = 0;
                on[(int64_t)bb * N + na] = 1;
                share[(int64_t)a * N + nb] = share[(int64_t)a * N + na];
                share[(int64_t)a * N + na] = 0.0;
                share[(int64_t)bb * N + na] = share[(int64_t)bb * N + nb];
                share[(int64_t)bb * N + nb] = 0.0;
                pieces[(int64_t)a * N + nb] = 1;
                pieces[(int64_t)a * N + na] = 0;
                pieces[(int64_t)bb * N + na] = 1;
                pieces[(int64_t)bb * N + nb] = 0;
                work[na] = work[na] - wa + wb;
                work[nb] = work[nb] - wb + wa;
                changed = 1;
            }
        }
        if (!changed) break;
    }

    /* 2. ranks, node by node */
    for (int32_t n = 0; n < N; ++n) {
        int32_t ni = 0;
        for (int32_t e = 0; e < E; ++e) {
            if (!on[(int64_t)e * N + n]) continue;
            int64_t k = pieces[(int64_t)e * N + n];
            for (int32_t c = 0; c < k; ++c) {
                struct plan_piece it = { share[(int64_t)e * N + n] / (double)k, e, c };
                int32_t p = ni++;
                while (p > 0 && piece_before(&it, &items[p - 1])) {
                    items[p] = items[p - 1];
                    --p;
                }
                items[p] = it;
            }
        }
        for (int32_t i = 0; i < g; ++i) rload[i] = 0.0;
        int32_t lim = (ni + g - 1) / g;
        if (lim > S) lim = S;
        int stuck = 0;
        for (int32_t t = 0; t < ni && !stuck; ++t) {
            int32_t b = -1;
            for (int32_t i = 0; i < g; ++i) {
                int32_t r = n * g + i;
                if (plan_used(slot_table, S, r) >= lim || plan_holds(slot_table, S, r, items[t].e))
                    continue;
                if (b < 0 || rload[i] < rload[b] ||
                    (rload[i] == rload[b] && plan_used(slot_table, S, r) <
                                             plan_used(slot_table, S, n * g + b)))
                    b = i;
            }
            if (b < 0) {
                stuck = 1;
                break;
            }
            int32_t r = n * g + b;
            slot_table[(int64_t)r * S + plan_used(slot_table, S, r)] = items[t].e;
            rload[b] += items[t].load;
            pl[(int64_t)items[t].e * G + r] += items[t].load;
        }
        if (stuck) {
            for (int32_t i = 0; i < g; ++i) {
                int32_t r = n * g + i;
                for (int32_t k = 0; k < S; ++k) slot_table[(int64_t)r * S + k] = -1;
                for (int32_t e = 0; e < E; ++e) pl[(int64_t)e * G + r] = 0.0;
            }
            int64_t kmax = 0;
            for (int32_t e = 0; e < E; ++e)
                if (on[(int64_t)e * N + n] && pieces[(int64_t)e * N + n] > kmax)
                    kmax = pieces[(int64_t)e * N + n];
            int32_t p = 0;
            for (int64_t k = kmax; k >= 1; --k)
                for (int32_t e = 0; e < E; ++e) {
                    if (!on[(int64_t)e * N + n] || pieces[(int64_t)e * N + n] != k) continue;
                    for (int64_t c = 0; c < k; ++c) {
                        int32_t r = n * g + p % g;
                        slot_table[(int64_t)r * S + plan_used(slot_table, S, r)] = e;
                        pl[(int64_t)e * G + r] += share[(int64_t)e * N + n] / (double)k;
                        ++p;
                    }
                }
        }
        /* repair: augmenting paths from the most loaded rank */
        for (int64_t moves = 0; moves < 4 * (int64_t)g * g * S; ++moves) {
            int32_t h = -1;
            double hl = 0.0;
            for (int32_t i = 0; i < g; ++i) {
                double l = plan_rank_load(pl, E, G, n * g + i);
                if (h < 0 || l > hl) {
                    h = i;
                    hl = l;
                }
            }
            if (!(hl > cap)) break;
            int32_t queue[32], parent[32], via[32];
            uint8_t seen[32] = { 0 };
            int32_t qh = 0, qt = 0, target = -1;
            queue[qt++] = h;
            seen[h] = 1;
            while (qh < qt && target < 0) {
                int32_t a = queue[qh++], ra = n * g + a;
                for (int32_t e = 0; e < E && target < 0; ++e) {
                    if (!(pl[(int64_t)e * G + ra] > 0.0)) continue;
                    for (int32_t b = 0; b < g && target < 0; ++b) {
                        int32_t rb = n * g + b;
                        if (seen[b]) continue;
                        if (!plan_holds(slot_table, S, rb, e) && plan_used(slot_table, S, rb) >= S)
                            continue;
                        seen[b] = 1;
                        parent[b] = a;
                        via[b] = e;
                        queue[qt++] = b;
                        if (plan_rank_load(pl, E, G, rb) < cap) target = b;
                    }
                }
            }
            if (target < 0) {
                /* slot swap: the heaviest expert eh on h (ties smaller e);
                   under-cap ranks u without a free slot and without eh, in
                   increasing load (ties smaller); on u, the expert x with
                   least work (ties smaller) that h does not hold and whose
                   work is below eh's on h. x moves whole to h, then
                   min(load_h - cap + w_x, cap - load_u + w_x, l_eh,h) of
                   eh moves to u. Needs a free slot on h. */
                int32_t rh = n * g + h;
                if (plan_used(slot_table, S, rh) >= S) break;
                int32_t eh = -1;
                for (int32_t k = 0; k < S; ++k) {
                    int32_t x = slot_table[(int64_t)rh * S + k];
                    if (x < 0) continue;
                    if (eh < 0 || pl[(int64_t)x * G + rh] > pl[(int64_t)eh * G + rh] ||
                        (pl[(int64_t)x * G + rh] == pl[(int64_t)eh * G + rh] && x < eh))
                        eh = x;
                }
                double weh = pl[(int64_t)eh * G + rh];
                int32_t bu = -1, bx = -1;
                double bul = 0.0;
                for (int32_t u = 0; u < g; ++u) {
                    int32_t ru = n * g + u;
                    double lu = plan_rank_load(pl, E, G, ru);
                    if (u == h || !(lu < cap) || plan_used(slot_table, S, ru) < S ||
                        plan_holds(slot_table, S, ru, eh))
                        continue;
                    int32_t x = -1;
                    for (int32_t k = 0; k < S; ++k) {
                        int32_t y = slot_table[(int64_t)ru * S + k];
                        if (y < 0 || plan_holds(slot_table, S, rh, y)) continue;
                        if (!(pl[(int64_t)y * G + ru] < weh)) continue;
                        if (x < 0 || pl[(int64_t)y * G + ru] < pl[(int64_t)x * G + ru] ||
                            (pl[(int64_t)y * G + ru] == pl[(int64_t)x * G + ru] && y < x))
                            x = y;
                    }
                    if (x < 0) continue;
                    if (bu < 0 || lu < bul) {
                        bu = u;
                        bx = x;
                        bul = lu;
                    }
                }
                if (bu < 0) break;
                int32_t ru = n * g + bu;
                double wx = pl[(int64_t)bx * G + ru];
                double mv = hl - cap + wx;
                if (cap - bul + wx < mv) mv = cap - bul + wx;
                if (weh < mv) mv = weh;
                if (!(mv > wx)) break;
                /* x: off u (slots stay packed), onto h */
                int32_t k = 0;
                while (slot_table[(int64_t)ru * S + k] != bx) ++k;
                for (; k + 1 < S; ++k) slot_table[(int64_t)ru * S + k] = slot_table[(int64_t)ru * S + k + 1];
                slot_table[(int64_t)ru * S + S - 1] = -1;
                slot_table[(int64_t)rh * S + plan_used(slot_table, S, rh)] = bx;
                pl[(int64_t)bx * G + ru] = 0.0;
                pl[(int64_t)bx * G + rh] += wx;
                /* part of eh: off h, onto u */
                slot_table[(int64_t)ru * S + plan_used(slot_table, S, ru)] = eh;
                pl[(int64_t)eh * G + rh] -= mv;
                pl[(int64_t)eh * G + ru] += mv;
                continue;
            }
            double mv = hl - cap;
            double room = cap - plan_rank_load(pl, E, G, n * g + target);
            if (room < mv) mv = room;
            for (int32_t b = target; b != h; b = parent[b]) {
                double avail = pl[(int64_t)via[b] * G + n * g + parent[b]];
                if (avail < mv) mv = avail;
            }
            if (!(mv > cap * 1e-12)) break;
            for (int32_t b = target; b != h; b = parent[b]) {
                int32_t e = via[b], ra = n * g + parent[b], rb = n * g + b;
                if (!plan_holds(slot_table, S, rb, e))
                    slot_table[(int64_t)rb * S + plan_used(slot_table, S, rb)] = e;
                pl[(int64_t)e * G + ra] -= mv;
                pl[(int64_t)e * G + rb] += mv;
            }
        }
        used[n] = 0;
        for (int32_t i = 0; i < g; ++i) used[n] += plan_used(slot_table, S, n * g + i);
    }

    /* 2b. global repair: augmenting paths over the ranks of all nodes */
    {
        int32_t* gq = (int32_t*)malloc((size_t)G * sizeof(int32_t));
        int32_t* gp = (int32_t*)malloc((size_t)G * sizeof(int32_t));
        int32_t* gv = (int32_t*)malloc((size_t)G * sizeof(int32_t));
        uint8_t* gs = (uint8_t*)malloc((size_t)G);
        if (!gq || !gp || !gv || !gs) {
            free(gq); free(gp); free(gv); free(gs);
            rc = REF_EINVAL;
            goto done;
        }
        for (int64_t moves = 0; moves < 4 * (int64_t)G * S; ++moves) {
            int32_t h = -1;
            double hl = 0.0;
            for (int32_t r = 0; r < G; ++r) {
                double l = plan_rank_load(pl, E, G, r);
                if (h < 0 || l > hl) {
                    h = r;
                    hl = l;
                }
            }
            if (!(hl > cap)) break;
            /* phase 0: through held replicas only; phase 1: also new
               replicas in free slots */
            int32_t target = -1;
            for (int32_t phase = 0; phase < 2 && target < 0; ++phase) {
                int32_t qh = 0, qt = 0;
                for (int32_t r = 0; r < G; ++r) gs[r] = 0;
                gq[qt++] = h;
                gs[h] = 1;
                while (qh < qt && target < 0) {
                    int32_t a = gq[qh++];
                    for (int32_t e = 0; e < E && target < 0; ++e) {
                        if (!(pl[(int64_t)e * G + a] > 0.0)) continue;
                        for (int32_t b = 0; b < G && target < 0; ++b) {
                            if (gs[b]) continue;
                            if (!plan_holds(slot_table, S, b, e) &&
                                (phase == 0 || plan_used(slot_table, S, b) >= S))
                                continue;
                            gs[b] = 1;
                            gp[b] = a;
                            gv[b] = e;
                            gq[qt++] = b;
                            if (cap - plan_rank_load(pl, E, G, b) > cap * 1e-12) target = b;
                        }
                    }
                }
            }
            if (target < 0) break;
            double mv = hl - cap;
            double room = cap - plan_rank_load(pl, E, G, target);
            if (room < mv) mv = room;
            for (int32_t b = target; b != h; b = gp[b]) {
                double avail = pl[(int64_t)gv[b] * G + gp[b]];
                if (avail < mv) mv = avail;
            }
            if (!(mv > cap * 1e-12)) break;
            for (int32_t b = target; b != h; b = gp[b]) {
                int32_t e = gv[b], nb = b / g;
                if (!plan_holds(slot_table, S, b, e)) {
                    slot_table[(int64_t)b * S + plan_used(slot_table, S, b)] = e;
                    on[(int64_t)e * N + nb] = 1;
                    used[nb] += 1;
                }
                pl[(int64_t)e * G + gp[b]] -= mv;
                pl[(int64_t)e * G + b] += mv;
            }
        }
        free(gq); free(gp); free(gv); free(gs);
    }

    /* 3. co-activation replicas */
    for (;;) {
        int32_t be = -1, bn = -1;
        int64_t bg = 0;
        for (int32_t e = 0; e < E; ++e)
            for (int32_t n = 0; n < N; ++n) {
                if (on[(int64_t)e * N + n] || used[n] >= all_slots) continue;
                int64_t gn = plan_gain(q, on, E, N, e, n);
                if (gn <= 0) continue;
                if (be < 0 || gn > bg || (gn == bg && count_ema[e] > count_ema[be])) {
                    be = e;
                    bn = n;
                    bg = gn;
                }
            }
        if (be < 0) break;
        int32_t b = -1;
        for (int32_t i = 0; i < g; ++i) {
            int32_t r = bn * g + i;
            if (plan_used(slot_table, S, r) >= S) continue;
            if (b < 0 || plan_used(slot_table, S, r) < plan_used(slot_table, S, bn * g + b)) b = i;
        }
        int32_t r = bn * g + b;
        slot_table[(int64_t)r * S + plan_used(slot_table, S, r)] = be;
        on[(int64_t)be * N + bn] = 1;
        used[bn] += 1;
    }

    /* owners, plan, objective, feasibility */
    for (int32_t e = 0; e < E; ++e) {
        owner[e] = -1;
        for (int32_t r = 0; r < G; ++r)
            if (plan_holds(slot_table, S, r, e) &&
                (owner[e] < 0 || pl[(int64_t)e * G + r] > pl[(int64_t)e * G + owner[e]]))
                owner[e] = r;
    }
    if (plan)
        for (int64_t i = 0; i < (int64_t)E * G; ++i) plan[i] = (float)pl[i];
    if (objective) {
        int64_t obj = 0;
        for (int32_t n = 0; n < N; ++n)
            for (int32_t i = 0; i < E; ++i)
                for (int32_t j = i + 1; j < E; ++j)
                    if (on[(int64_t)i * N + n] && on[(int64_t)j * N + n]) obj += q[(int64_t)i * E + j];
        *objective = (double)obj / 256.0;
    }
    if (feasible) {
        int ok = 1;
        for (int32_t r = 0; r < G; ++r)
            if (plan_rank_load(pl, E, G, r) > cap * (1.0 + 1e-9)) ok = 0;
        *feasible = ok;
    }
done:
    free(q); free(on); free(share); free(pieces); free(order); free(used); free(work); free(pl);
    free(items); free(rload); free(dest);
    return rc;
}

int ref_plan_layout(int32_t N, int32_t g, int32_t E, int32_t S, const float* coact_ema,
                    const float* count_ema, float eps, int32_t* slot_table, int32_t* owner,
                    float* plan, double* objective, int32_t* feasible)
{
    /* node fill fractions of step 1 and 1b after the first */
    static const double retry[3] = { 0.98, 0.95, 0.90 };
    int32_t ok = 0;
    int rc = plan_once(N, g, E, S, coact_ema, count_ema, eps, 1.0, slot_table, owner, plan,
                       objective, &ok);
    if (rc != REF_OK || ok) {
        if (rc == REF_OK && feasible) *feasible = ok;
        return rc;
    }
    int32_t G = N * g;
    int32_t* t2 = (int32_t*)malloc((size_t)G * S * sizeof(int32_t));
    int32_t* o2 = (int32_t*)malloc((size_t)E * sizeof(int32_t));
    float* p2 = (float*)malloc((size_t)E * G * sizeof(float));
    if (!t2 || !o2 || !p2) {
        free(t2); free(o2); free(p2);
        return REF_EINVAL;
    }
    for (int k = 0; k < 3 && !ok; ++k) {
        double obj2 = 0.0;
        int32_t ok2 = 0;
        if (plan_once(N, g, E, S, coact_ema, count_ema, eps, retry[k], t2, o2, p2, &obj2, &ok2) !=
                REF_OK ||
            !ok2)
            continue;
        memcpy(slot_table, t2, (size_t)G * S * sizeof(int32_t));
        memcpy(owner, o2, (size_t)E * sizeof(int32_t));
        if (plan) memcpy(plan, p2, (size_t)E * G * sizeof(float));
        if (objective) *objective = obj2;
        ok = 1;
    }
    free(t2); free(o2); free(p2);
    if (feasible) *feasible = ok;
    return REF_OK;
}

/* ---------------------------------------------------------------------- */
/* Stage 1 (Section 3.2, Eq. 3) solved exactly, for tiny instances only    */
/* (E <= 6 experts, G <= 4 ranks). Every layout is visited: rank r takes a */
/* set P_r of at most S experts (a bitmask over the experts), ranks in     */
/* order and sets in increasing mask value. A layout counts if every       */
/* expert has a replica and a division of the work exists; its value is    */
/* Eq. 3's objective, the sum of c_ij over the pairs i < j whose experts   */
/* both have a replica on a node, once for each such node. The first       */
/* layout of the highest value is returned.                                */
/*                                                                         */
/* A division {w'_er} (w'_er >= 0, zero where e is not on r, sum_r w'_er = */
/* w_e, sum_e w'_er <= cap on every rank) exists exactly when every set A  */
/* of experts fits on the ranks that hold any of them:                     */
/*     sum_{e in A} w_e <= cap * |{r : P_r meets A}|,                      */
/* the supply-demand theorem for bipartite transport (Gale 1957), i.e.     */
/* max-flow = min-cut on source -> e (capacity w_e) -> r (if e is on r,    */
/* unbounded) -> sink (capacity cap). cap = (1 + eps) * sum_e w_e / G is   */
/* the balance bound of Eq. 3 with the planned work in place of KT. A set  */
/* fits when its work exceeds the bound by at most a relative 1e-9.        */
/* Pair weights are read as given (only c_ij with i < j).                  */
/* ---------------------------------------------------------------------- */
struct exact_ctx {
    int32_t N, g, E, S, G;
    const float* c;
    double w[6];
    double cap;
    uint32_t cur[4];   /* P_r of the layout being visited */
    uint32_t best_layout[4];
    double best;
    int found;
};

static double exact_value(const struct exact_ctx* x)
{
    double v = 0.0;
    for (int32_t n = 0; n < x->N; ++n) {
        uint32_t on = 0; /* experts with a replica on node n */
        for (int32_t i = 0; i < x->g; ++i) on |= x->cur[n * x->g + i];
        for (int32_t a = 0; a < x->E; ++a)
            for (int32_t b = a + 1; b < x->E; ++b)
                if ((on >> a & 1u) && (on >> b & 1u)) v += (double)x->c[a * x->E + b];
    }
    return v;
}

static int exact_divisible(const struct exact_ctx* x)
{
    for (uint32_t A = 1; A < (1u << x->E); ++A) {
        double need = 0.0;
        int32_t holders = 0;
        for (int32_t e = 0; e < x->E; ++e)
            if (A >> e & 1u) need += x->w[e];
        for (int32_t r = 0; r < x->G; ++r)
            if (x->cur[r] & A) ++holders;
        if (need > x->cap * (double)holders * (1.0 + 1e-9)) return 0;
    }
    return 1;
}

static void exact_visit(struct exact_ctx* x, int32_t r)
{
    if (r == x->G) {
        uint32_t all = 0;
        for (int32_t k = 0; k < x->G; ++k) all |= x->cur[k];
        if (all != (1u << x->E) - 1u) return; /* an expert without a replica */
        double v = exact_value(x);
        if (x->found && !(v > x->best)) return; /* cannot replace the first best */
        if (!exact_divisible(x)) return;
        x->best = v;
        memcpy(x->best_layout, x->cur, sizeof(x->cur));
        x->found = 1;
        return;
    }
    for (uint32_t m = 0; m < (1u << x->E); ++m) {
        if (popcount32(m) > x->S) continue;
        x->cur[r] = m;
        exact_visit(x, r + 1);
    }
}

/* Outputs: *found = 1 if some layout meets every constraint (else 0 and
 * nothing else is written); *objective its value; slot_table [G][S] the
 * first best layout, each rank's experts in increasing id, -1 after. */
int ref_plan_exact(int32_t N, int32_t g, int32_t E, int32_t S, const float* coact,
                   const float* work, float eps, int32_t* found, double* objective,
                   int32_t* slot_table)
{
    if (N < 1 || g < 1 || N * g > 4 || E < 1 || E > 6 || S < 1 || !coact || !work || !found)
        return REF_EINVAL;
    if (!(eps >= 0.0f)) return REF_EINVAL;
    struct exact_ctx x;
    memset(&x, 0, sizeof(x));
    x.N = N;
    x.g = g;
    x.E = E;
    x.S = S;
    x.G = N * g;
    x.c = coact;
    double total = 0.0;
    for (int32_t e = 0; e < E; ++e) {
        if (!(work[e] >= 0.0f) || isinf(work[e])) return REF_EINVAL;
        x.w[e] = (double)work[e];
        total += x.w[e];
    }
    x.cap = (1.0 + (double)eps) * total / (double)x.G;
    exact_visit(&x, 0);
    *found = x.found;
    if (!x.found) return REF_OK;
    if (objective) *objective = x.best;
    if (slot_table) {
        for (int32_t r = 0; r < x.G; ++r) {
            int32_t k = 0;
            for (int32_t e = 0; e < E; ++e)
                if (x.best_layout[r] >> e & 1u) slot_table[r * S + k++] = e;
            for (; k < S; ++k) slot_table[r * S + k] = -1;
        }
    }
    return REF_OK;
}
