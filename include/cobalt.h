/*
 * cobalt.h - C ABI of the co-activation token-routing path of Cobalt
 * ("Leveraging Expert Co-activation for Efficient Distributed MoE Training").
 *
 * One MoE layer, one training step, on one GPU. G = N * gpus_per_node
 * virtual ranks on N virtual nodes; node(r) = r / gpus_per_node. T tokens,
 * each with K selected experts out of E (topk_idx[t][j], slot j). Pair
 * p = t*K + j is the task (t, topk_idx[t][j]).
 *
 * Conventions for every call below:
 *  - Pointers are DEVICE pointers unless the name starts with host_.
 *  - Arrays are dense, row-major, in the element type of the declaration;
 *    bf16 rows are raw 16-bit patterns, 16-byte aligned.
 *  - The caller owns every buffer. The four path calls (cobalt_coact_stats,
 *    cobalt_assign, cobalt_dispatch_pack, cobalt_combine) allocate nothing,
 *    enqueue their kernels on `stream` (a hipStream_t; NULL = the default
 *    stream of the current device) and return without synchronising.
 *  - Errors are reported by return code only. Argument checks run on the
 *    host before anything is enqueued; on any error nothing is enqueued and
 *    no output is touched. Data-dependent checks (expert ids in range,
 *    distinct experts per token, non-decreasing source ranks) are made only
 *    by cobalt_validate_routing: on data that fails them the path calls do
 *    not read or write outside the buffers they were given, but their
 *    results are unspecified (except where a call states them, as
 *    cobalt_coact_stats does for repeated and out-of-range ids).
 *  - Calls on distinct (layout, stream, output buffers) may run concurrently.
 */
#ifndef COBALT_H
#define COBALT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    COBALT_OK = 0,
    COBALT_EINVAL = 1,       /* bad argument (null pointer, size out of range, misaligned) */
    COBALT_EUNSUPPORTED = 2, /* valid request outside the library's limits */
    COBALT_ENOMEM = 3,       /* device allocation failed (layout calls only) */
    COBALT_EHIP = 4,         /* a HIP runtime call or kernel launch failed */
    COBALT_EDATA = 5         /* input data violates the model (layout or routing) */
} cobalt_status;

/* Limits of the library: 1 <= N <= 16, 1 <= gpus_per_node <= 32,
 * G = N * gpus_per_node <= 512, 1 <= K <= 16, 1 <= E <= 4096,
 * T * K < 2^31, d % 8 == 0 (rows are whole 16-byte vectors). */

const char* cobalt_status_string(cobalt_status s);

/* ------------------------------------------------------------------------
 * Expert layout {P_r} (Section 3.1, "Problem formulation"; the per-expert
 * sets R_{e,n} and N_e of Section 3.3, step 1).
 *
 * host_slot_table [G][S]: expert ids held by rank r, -1 = empty slot.
 * host_owner_rank [E]:    owner rank of each expert (used by the owner-only
 *                         baseline of cobalt_assign), or NULL = the lowest
 *                         rank holding the expert.
 * The layout is rejected with COBALT_EDATA if an expert has no replica
 * (coverage constraint of Eq. 2), a rank holds an expert twice (placement
 * rule of Section 3.2, Stage 2), an owner does not hold its expert, or an
 * id lies outside [-1, E). The slot budget S = (1+rho)E/G of Eq. 2 is the
 * table's width.
 * Derives node_mask[e] (bit n: e on node n) and rank_mask[e][n] (bit i: e
 * on rank n*g+i) and copies them, with the owners, to the current device.
 * Synchronous; the handle belongs to the device current at creation and may
 * only be used there.
 * ---------------------------------------------------------------------- */
typedef struct cobalt_layout_s* cobalt_layout_t;

cobalt_status cobalt_layout_create(int32_t N, int32_t gpus_per_node, int32_t E, int32_t S,
                                   const int32_t* host_slot_table,
                                   const int32_t* host_owner_rank,
                                   cobalt_layout_t* out);
cobalt_status cobalt_layout_destroy(cobalt_layout_t layout);

/* Copies the derived tables back to the host (synchronous): node_mask [E],
 * rank_mask [E][N], owner_rank [E]. Any output may be NULL. */
cobalt_status cobalt_layout_tables(cobalt_layout_t layout, uint32_t* host_node_mask,
                                   uint32_t* host_rank_mask, int32_t* host_owner_rank);

/* ------------------------------------------------------------------------
 * Step 1: co-activation statistics (Section 3.2, Stage 1: c_ij counts the
 * tokens that select both experts i and j; w_e counts the tasks of e).
 *
 * topk_idx [T][K] int32 in, coact [E][E] uint32 in/out, expert_count [E]
 * uint32 in/out (may be NULL).
 * For every token and every ordered pair of distinct slots (a, b):
 * coact[topk_idx[t][a]][topk_idx[t][b]] += 1; for every slot:
 * expert_count[topk_idx[t][a]] += 1. Nothing is zeroed: counts accumulate
 * across calls (and steps) until the caller clears them. With distinct
 * experts per token coact is symmetric with a zero diagonal and row sums
 * (K-1) * expert_count; an expert a token holds m times adds m(m-1) to
 * its diagonal entry. Ids outside [0, E) count nowhere.
 * K > E is rejected with COBALT_EINVAL (a token's experts are distinct).
 * workspace: device scratch of at least cobalt_coact_stats_workspace_bytes(
 *   T, K, E) bytes (partial histograms of E(E-1)/2 bins for each chunk of
 *   about 1024 tokens, at most 128 chunks; 2 bytes per bin where a chunk's
 *   bins cannot pass 65535, else 4), 256-byte aligned, owned by the
 *   caller; contents on entry are ignored; it must not be shared by calls
 *   that may overlap. The call updates coact and expert_count with plain
 *   (non-atomic) adds, or with integer atomic adds when it is small (at most
 *   65536 bin updates) and on the diagonal, so calls that may overlap must
 *   not share them either. The counts are exact either way and do not
 *   depend on scheduling.
 * ---------------------------------------------------------------------- */
size_t cobalt_coact_stats_workspace_bytes(int64_t T, int32_t K, int32_t E);

cobalt_status cobalt_coact_stats(const int32_t* topk_idx, int64_t T, int32_t K, int32_t E,
                                 uint32_t* coact, uint32_t* expert_count,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Step 2: communication-aware task assignment (Section 3.3, Algorithm 1).
 *
 * topk_idx [T][K] int32 in; src_rank [T] int32 in, the source rank s_t of
 * each token, non-decreasing, or NULL = contiguous blocks s_t = t / (T/G)
 * (then T % G must be 0).
 * mode 0 = Algorithm 1: the experts held on the source node run there; the
 *   rest are covered by the fewest remote nodes (the first cover in order of
 *   (node count, remote-node bitmask), where remote bit i is the i-th node
 *   other than node(s_t)); each such expert draws one of the chosen nodes
 *   holding it, then every task draws one rank of its node holding the
 *   expert. No load cap is applied.
 * mode 1 = owner-only baseline: every task runs on its expert's owner rank.
 * K above the layout's E is rejected with COBALT_EINVAL.
 * Draws are counter-based: with sm(z) the SplitMix64 output for state z
 * (Steele, Lea & Flood 2014), key = sm(sm(seed) ^ step),
 * h = sm(key ^ (p << 1 | s)) for pair p and draw s (0 = node, 1 = rank),
 * and the drawn index among c candidates (set bits, ascending) is
 * ((h >> 32) * c) >> 32.
 * assigned_rank [T][K] int32 out: r_te per pair. remote_nodes [T] uint16
 * out (may be NULL): bit n set iff node n != node(s_t) receives token t
 * (its popcount is the token's term of Eq. 1).
 * ---------------------------------------------------------------------- */
cobalt_status cobalt_assign(cobalt_layout_t layout, const int32_t* topk_idx,
                            const int32_t* src_rank, int64_t T, int32_t K,
                            uint64_t seed, uint64_t step, int32_t mode,
                            int32_t* assigned_rank, uint16_t* remote_nodes, void* stream);

/* ------------------------------------------------------------------------
 * Step 3: dispatch layout and pack (the EP dispatch all-to-all's send side,
 * Section 1 and Fig. 1; here one row per (token, expert) pair).
 *
 * Bucket of pair p: (s_t, r_p). Buckets are laid out in row-major order
 * (per-source send buffers, each split by destination rank), and each
 * bucket keeps its pairs in increasing p.
 * assigned_rank [T][K] int32 in; src_rank as in cobalt_assign;
 * x [T][d] bf16 in (may be NULL together with packed: layout only).
 * send_counts [G][G] int32 out: pairs per (source, destination).
 * send_offsets [G*G+1] int64 out: exclusive prefix sum of send_counts,
 *   send_offsets[G*G] = number of pairs placed (T*K on valid data).
 * pos [T][K] int32 out: packed row of each pair.
 * packed [T*K][d] bf16 out: packed[pos[p]] = x[t], bit for bit.
 * workspace: device scratch of at least cobalt_dispatch_workspace_bytes(T,
 *   K, G) bytes, 256-byte aligned, owned by the caller; contents on entry
 *   are ignored; it must not be shared by calls that may overlap.
 * ---------------------------------------------------------------------- */
size_t cobalt_dispatch_workspace_bytes(int64_t T, int32_t K, int32_t G);

cobalt_status cobalt_dispatch_pack(const int32_t* assigned_rank, const int32_t* src_rank,
                                   int64_t T, int32_t K, int32_t G,
                                   const void* x, int64_t d,
                                   int32_t* send_counts, int64_t* send_offsets,
                                   int32_t* pos, void* packed,
                                   void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Step 3 without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc and its like).
 *
 * Same arguments, outputs and errors as cobalt_dispatch_pack, less the
 * workspace: its place is taken by a fixed scratch array of
 * COBALT_DISPATCH_NOALLOC_SCRATCH_BYTES bytes in the library's device
 * memory. Each GPU the library runs on holds its own copy from when the
 * library's code is loaded there until the process ends. The call allocates
 * nothing; its first call on a device only looks up that device's copy.
 * Returns COBALT_EUNSUPPORTED, before anything is enqueued, when
 * cobalt_dispatch_workspace_bytes(T, K, G) exceeds the array (with G = 64
 * that is above 66 973 696 pairs T*K; with G = 512, above 7 335 936).
 * Every call on one GPU uses that GPU's one array, and the array keeps what
 * the last call left in it (each call re-initialises what it reads), so
 * calls that may overlap on one GPU (different streams, or host threads
 * without ordering) race and give wrong results: issue them on one stream,
 * or order them. Calls on different GPUs do not interact.
 * ---------------------------------------------------------------------- */
#define COBALT_DISPATCH_NOALLOC_SCRATCH_BYTES ((size_t)8 << 20)

cobalt_status cobalt_dispatch_pack_noalloc(const int32_t* assigned_rank, const int32_t* src_rank,
                                           int64_t T, int32_t K, int32_t G,
                                           const void* x, int64_t d,
                                           int32_t* send_counts, int64_t* send_offsets,
                                           int32_t* pos, void* packed, void* stream);

/* ------------------------------------------------------------------------
 * Step 3': node-deduplicated dispatch layout and pack (Section 1 and
 * Section 3.1, Eq. 1: a token crosses to a node once, however many ranks
 * there need it, and is then forwarded inside the node).
 *
 * Token t has one row per distinct node n among { node(r_tj) }, its own
 * node included, so the rows whose node differs from node(s_t) number
 * exactly Eq. 1's V. Bucket of row (t, n): (s_t, n), buckets in row-major
 * order over [G][N]; each bucket keeps its rows in increasing t.
 * assigned_rank [T][K] int32 in; src_rank as in cobalt_assign; G = N *
 *   gpus_per_node.
 * x [T][d] bf16 in (may be NULL together with packed: layout only).
 * node_counts [G][N] int32 out: rows per (source rank, destination node).
 * node_offsets [G*N+1] int64 out: exclusive prefix sum of node_counts,
 *   node_offsets[G*N] = number of rows.
 * node_pos [T][N] int32 out: row of (t, n), -1 if no slot of t goes to n.
 * fwd_mask [rows] uint32 out: the intra-node forwarding index; bit i is set
 *   iff some slot of the row's token is assigned to rank n*gpus_per_node+i.
 * row_token [rows] int32 out (may be NULL): token of each row.
 * packed [rows][d] bf16 out: packed[node_pos[t][n]] = x[t], bit for bit.
 * fwd_mask, row_token and packed must hold T * min(K, N) rows, the most a
 *   call can produce.
 * workspace: device scratch of at least
 *   cobalt_node_dispatch_workspace_bytes(T, N, gpus_per_node) bytes,
 *   256-byte aligned, owned by the caller; contents on entry are ignored;
 *   it must not be shared by calls that may overlap.
 * Slots with a rank outside [0, G) are skipped; such data is rejected by
 * cobalt_validate_routing.
 * ---------------------------------------------------------------------- */
size_t cobalt_node_dispatch_workspace_bytes(int64_t T, int32_t N, int32_t gpus_per_node);

cobalt_status cobalt_node_dispatch_pack(const int32_t* assigned_rank, const int32_t* src_rank,
                                        int64_t T, int32_t K, int32_t N, int32_t gpus_per_node,
                                        const void* x, int64_t d,
                                        int32_t* node_counts, int64_t* node_offsets,
                                        int32_t* node_pos, uint32_t* fwd_mask,
                                        int32_t* row_token, void* packed,
                                        void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Step 4: combine and weighted sum (Fig. 1, last stage).
 *
 * expert_out [T*K][d] bf16 in, in the packed layout (row pos[p] holds the
 * result of pair p); pos [T][K] int32 in; gates [T][K] fp32 in.
 * y [T][d] bf16 out:
 *   y[t][c] = bf16_rne( sum_{j=0..K-1} gates[t][j] * expert_out[pos[t][j]][c] )
 * accumulated in fp32 from 0 with one fused multiply-add per slot in slot
 * order. y_f32 [T][d] fp32 out (may be NULL) receives the fp32 sums. A pos
 * outside [0, T*K) contributes nothing.
 * ---------------------------------------------------------------------- */
cobalt_status cobalt_combine(const void* expert_out, const int32_t* pos, const float* gates,
                             int64_t T, int32_t K, int64_t d,
                             void* y, float* y_f32, void* stream);

/* ------------------------------------------------------------------------
 * Step 4': node-level combine, the reverse of the node-deduplicated
 * dispatch (Section 1 and Section 3.1: a token's results leave a node once,
 * so the combine's cross-node rows also number Eq. 1's V).
 *
 * On node n the slots of token t whose rank lies on n are summed first:
 *   part[t][n][c] = bf16_rne( sum_{j : r_tj / gpus_per_node = n}
 *                             gates[t][j] * expert_out[pos[t][j]][c] ),
 * in fp32 from 0 with one fused multiply-add per slot in slot order. The
 * partial is stored as bf16, like the rows of the dispatch, in row
 * node_pos[t][n] of node_partial, the row the node-deduplicated dispatch
 * used for (t, n). At the source the partials are summed in increasing n:
 *   y[t][c] = bf16_rne( sum_{n : node_pos[t][n] >= 0} float(part[t][n][c]) ),
 * in fp32 from 0.
 * expert_out [T*K][d] bf16 in, in the per-pair packed layout; pos [T][K]
 *   int32 in (from cobalt_dispatch_pack); assigned_rank [T][K] int32 in;
 *   gates [T][K] fp32 in; node_pos [T][N] int32 in (from
 *   cobalt_node_dispatch_pack on the same assigned_rank and src_rank).
 * node_partial [T*min(K,N)][d] bf16 out: only the rows that node_pos names
 *   are written. y [T][d] bf16 out.
 * G = N * gpus_per_node. A slot is skipped if its rank is outside [0, G)
 *   or its row outside [0, T*K); a node_pos entry outside
 *   [0, T*min(K,N)) is neither written nor summed. A named node row with
 *   no slot of its token on the node is written as zero.
 * The result differs from cobalt_combine by the rounding of the partials
 *   to bf16 (with a single node it is identical).
 * ---------------------------------------------------------------------- */
cobalt_status cobalt_node_combine(const void* expert_out, const int32_t* pos,
                                  const int32_t* assigned_rank, const float* gates,
                                  const int32_t* node_pos, int64_t T, int32_t K, int32_t N,
                                  int32_t gpus_per_node, int64_t d, void* node_partial, void* y,
                                  void* stream);

/* ------------------------------------------------------------------------
 * Per-replica workload (Section 3.1 workload model: w_er counts the tasks of
 * expert e executed on rank r; Section 3.2, Stage 2 tracks it per replica).
 *
 * topk_idx [T][K] int32 in, assigned_rank [T][K] int32 in (the output of
 * cobalt_assign), load [E][G] uint32 in/out:
 *   load[e][r] += #{(t, j) : topk_idx[t][j] = e and assigned_rank[t][j] = r}.
 * Pairs with an id outside [0, E) or a rank outside [0, G) are skipped.
 * Nothing is zeroed (counts accumulate). workspace: device scratch of at
 * least cobalt_replica_load_workspace_bytes(T, K, E, G) bytes, 256-byte
 * aligned, owned by the caller, contents ignored, not shared by calls that
 * may overlap; load is updated with plain adds, so overlapping calls must
 * not share it either.
 * ---------------------------------------------------------------------- */
size_t cobalt_replica_load_workspace_bytes(int64_t T, int32_t K, int32_t E, int32_t G);

cobalt_status cobalt_replica_load(const int32_t* topk_idx, const int32_t* assigned_rank,
                                  int64_t T, int32_t K, int32_t E, int32_t G, uint32_t* load,
                                  void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Per-step intra-node rebalancing (Section 3.2, Stage 2). Host only,
 * synchronous, no device memory.
 *
 * host_slot_table [G][S] in (as in cobalt_layout_create); host_owner_rank
 * [E] in or NULL (= lowest rank holding the expert); host_replica_load
 * [E][G] in: estimated workload of the replica of e on rank r (finite,
 * >= 0; entries without a replica are ignored).
 * For each node, the replicas on the node's ranks are sorted by load
 * (heaviest first; ties by expert id, then by previous rank) and placed one
 * by one on the least-loaded rank of that node (ties: lowest rank) that has
 * a free slot and no replica of the same expert. The set of replicas per
 * node is unchanged. If some replica finds no eligible rank, the node keeps
 * its previous placement.
 * host_new_slot_table [G][S] out (may alias nothing else); host_new_owner_rank
 * [E] out or NULL: the rank the owner replica moved to; host_rank_load [G]
 * out or NULL: the summed replica load of each rank after placement, in
 * placement order (fp32).
 * Returns COBALT_EDATA for an invalid table, owner or load.
 * ---------------------------------------------------------------------- */
cobalt_status cobalt_intra_node_rebalance(int32_t N, int32_t gpus_per_node, int32_t E, int32_t S,
                                          const int32_t* host_slot_table,
                                          const int32_t* host_owner_rank,
                                          const float* host_replica_load,
                                          int32_t* host_new_slot_table,
                                          int32_t* host_new_owner_rank, float* host_rank_load);

/* ------------------------------------------------------------------------
 * Periodic global planning (Section 3.2, Stage 1; Eq. 3), host only.
 *
 * Chooses a replica layout and a division of each expert's estimated work
 * over its replicas that keep co-activated experts on the same node:
 * maximise sum_n sum_{i<j} c_ij [i and j both on node n] with every expert
 * placed, at most S replicas per rank, no expert twice on a rank, and at
 * most cap = (1 + eps) W / G planned work per rank, W = sum_e w_e. The
 * paper solves this as a MILP; this is a deterministic greedy heuristic for
 * the same objective and constraints (work placement on nodes by longest
 * processing time, moves and swaps that raise the objective, rank packing
 * with augmenting-path repair of the work division inside each node and
 * then across nodes, then replicas that raise the objective in the
 * remaining slots; a plan above the cap is made again with work slack left
 * on every node). Pair weights are quantised to 1/256 so that every
 * comparison of gains is exact.
 *
 * host_coact_ema [E][E] fp32 in: c_ij (EMA of co-activation counts; only
 *   i < j is read; finite, >= 0, <= 2^28, so that every integer sum of the
 *   quantised weights fits in int64).
 * host_count_ema [E] fp32 in: w_e (EMA of expert task counts; finite, >= 0).
 * eps: the allowed imbalance (>= 0; the paper's default is 0.15).
 * host_slot_table [G][S] int32 out: expert ids, -1 for empty slots.
 * host_owner_rank [E] int32 out: the rank with the most planned work.
 * host_plan [E][G] fp32 out (may be NULL): planned work w'_er, which can
 *   initialise Stage 2's replica-level EMA.
 * host_objective (may be NULL): the objective, from the quantised weights.
 * host_feasible (may be NULL): 1 if every rank's planned work is within
 *   cap (1 + 1e-9), else 0 (the heuristic found no division within cap).
 * Returns COBALT_EINVAL for bad sizes, G*S < E or a bad eps, COBALT_EDATA
 * for bad statistics or when some expert finds no free slot.
 * ---------------------------------------------------------------------- */
cobalt_status cobalt_plan_layout(int32_t N, int32_t gpus_per_node, int32_t E, int32_t S,
                                 const float* host_coact_ema, const float* host_count_ema,
                                 float eps, int32_t* host_slot_table, int32_t* host_owner_rank,
                                 float* host_plan, double* host_objective,
                                 int32_t* host_feasible);

/* ------------------------------------------------------------------------
 * Planner statistics (Section 3.2): exponential moving averages of the
 * step's counts, and the Ochiai similarity of expert pairs (Section 1, the
 * footnote on Fig. 3). The paper gives no decay; it is a parameter.
 *
 * One EMA update of m with a count x, in fp32:
 *   COBALT_EMA_INIT set:  m = x
 *   otherwise:            m = fma(decay, m, (1 - decay) * x)
 * with x the count rounded to fp32 and 1 - decay rounded to fp32 once.
 * COBALT_EMA_CLEAR set: the counts are set to 0 after they are read, so the
 * next step's statistics start from zero with no separate clearing call.
 * decay must lie in [0, 1]; flags other than these two bits are rejected.
 * ---------------------------------------------------------------------- */
#define COBALT_EMA_INIT 1
#define COBALT_EMA_CLEAR 2

/* Stage 1's statistics: EMAs of c_ij and w_e from the counts of
 * cobalt_coact_stats, and the Ochiai similarity of the step's counts.
 * coact [E][E] uint32 in (cleared with COBALT_EMA_CLEAR); expert_count [E]
 * uint32 in (cleared likewise).
 * ema_coact [E][E] fp32 in/out (may be NULL); ema_count [E] fp32 in/out (may
 * be NULL); ochiai [E][E] fp32 out (may be NULL):
 *   ochiai[i][j] = coact[i][j] / sqrt(expert_count[i] * expert_count[j]),
 *   ochiai[i][i] = 1 for an expert with a nonzero count,
 * and 0 where the pair shares no token or either count is 0, each
 * operation one correctly rounded fp32 operation. */
cobalt_status cobalt_coact_ema(uint32_t* coact, uint32_t* expert_count, int32_t E, float decay,
                               int32_t flags, float* ema_coact, float* ema_count, float* ochiai,
                               void* stream);

/* EMA of any n uint32 counts, e.g. Stage 2's replica-level w_er from
 * cobalt_replica_load (initialised by the caller, e.g. from the planned
 * workload division, before the first update). counts [n] uint32 in (cleared
 * with COBALT_EMA_CLEAR); ema [n] fp32 in/out (may be NULL to clear only). */
cobalt_status cobalt_count_ema(uint32_t* counts, int64_t n, float decay, int32_t flags,
                               float* ema, void* stream);

/* ------------------------------------------------------------------------
 * Debug check of routing inputs (synchronous; allocates a few bytes).
 * Checks 0 <= topk_idx < E, distinct experts within each token, and, if
 * src_rank is given, 0 <= src_rank < G and non-decreasing. Returns COBALT_OK
 * or COBALT_EDATA; host_flags (may be NULL) receives a bitmask:
 * 1 = expert id out of range, 2 = duplicate expert in a token,
 * 4 = source rank out of range, 8 = source ranks decreasing.
 * ---------------------------------------------------------------------- */
cobalt_status cobalt_validate_routing(const int32_t* topk_idx, const int32_t* src_rank,
                                      int64_t T, int32_t K, int32_t E, int32_t G,
                                      uint32_t* host_flags, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* COBALT_H */
