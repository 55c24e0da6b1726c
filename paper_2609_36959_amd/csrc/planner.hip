// Periodic global planning (Section 3.2, Stage 1), host side.
//
// Eq. 3 chooses the replica layout {P_r} and a division w'_er of each
// expert's estimated work w_e over its replicas to maximise the
// co-activation inside nodes, sum_n sum_{i<j} c_ij [i and j both on n],
// with every expert placed, at most S replicas per rank, no expert twice on
// a rank, and at most cap = (1 + eps) W / G planned work per rank (W =
// sum_e w_e). The paper solves its MILP form with a MILP solver; this is a
// deterministic greedy heuristic for the same problem:
//
//   q_ij = llrint(256 c_ij) (int64), so every gain is an exact integer sum;
//   gain(e, n) = sum of q_ex over the other experts x on node n;
//   need(x) = 1 if x <= cap, else ceil(x / cap) (ranks a share x needs).
//
//   1. Work placement: experts by decreasing w (ties: smaller id) take
//      nodes one at a time, best first by (the remainder fits in the node's
//      spare work g cap - work and free slots, spare work left, spare work,
//      gain), ties to the smaller node; nodes first keep R = min(g, (G S -
//      sum_e need(w_e)) / N) slots free for step 2, and give them up only
//      when no node qualifies or only a node using them fits. A share uses
//      need(share) slots (at most the node's free slots and g).
//   1b. Local search: sweeps over the experts placed whole in one slot of
//      one node ("single"), in increasing id, apply for each the best
//      improving move to a node with a free slot or swap with a single
//      expert of another node (ties: moves first, then smaller node or
//      partner), keeping every changed node within g cap or not above its
//      previous work; until a sweep changes nothing (at most 64 sweeps).
//   2. Ranks per node: shares cut into need equal pieces go, in decreasing
//      work (ties: smaller e, earlier piece), to the least-loaded rank
//      (ties: fewer replicas, smaller rank) with fewer than min(S,
//      ceil(pieces / g)) replicas and without the expert; if a piece finds
//      none, the node is laid out round-robin instead. Repair: while the
//      most loaded rank h exceeds cap, push work along the shortest
//      augmenting path of expert -> rank edges (a rank holding the expert,
//      or with a free slot for a new replica) to the first rank found
//      below cap; with no such path, a slot swap moves a light expert from
//      a full under-cap rank to h and part of h's heaviest expert into the
//      freed slot.
//   2b. Global repair: the same augmenting-path search over the ranks of all
//      nodes, so that a node left above its ranks' caps passes work to
//      another node: first through ranks that hold the path's expert, and
//      only if that reaches no target through free slots too (a new replica
//      makes its expert a member of that node). A target needs room above
//      cap 1e-12; at most 4 G S moves.
//   3. Co-activation replicas: while a node has a free slot, add the
//      (e, n) with the largest positive gain (ties: larger w, smaller e,
//      smaller n), with no planned work, on the node's rank with fewest
//      replicas (ties: smaller).
//   owner[e]: the rank with the most planned work for e (ties: smaller).
//   Retries: a plan above the cap is made again with the node work bound of
//   steps 1 and 1b at f g cap, f = 0.98, 0.95, 0.90 in turn (slack on every
//   node for steps 2 and 2b); the first plan within the cap is returned, and
//   if none is, the plan with f = 1.
//
// Rank loads are always summed over the rank's experts in increasing id, so
// every floating-point decision is reproducible.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "internal.hpp"

namespace cobalt {
namespace {

struct Planner {
    int N, g, G, E, S;
    double cap = 0.0, node_cap = 0.0;
    int64_t all_slots = 0, node_slots = 0;
    const float* w;
    std::vector<int64_t> q;     // [E][E], upper triangle used
    std::vector<int64_t> gain;  // [E][N]
    std::vector<uint8_t> on;    // [E][N]
    std::vector<double> share;  // [E][N]
    std::vector<int64_t> pieces;  // [E][N]
    std::vector<int64_t> used;  // [N] slots counted by steps 1 and 1b, then actual
    std::vector<double> work;   // [N]
    std::vector<std::vector<int32_t>> slots;  // [G], in placement order
    std::vector<double> pl;     // [E][G]

    int64_t qq(int a, int b) const {
        if (a == b) return 0;
        return a < b ? q[(size_t)a * E + b] : q[(size_t)b * E + a];
    }
    int64_t need(double x) const { return x <= cap ? 1 : (int64_t)std::ceil(x / cap); }

    void join(int e, int n) {  // e becomes a member of node n
        on[(size_t)e * N + n] = 1;
        for (int x = 0; x < E; ++x) gain[(size_t)x * N + n] += qq(x, e);
    }
    void leave(int e, int n) {
        on[(size_t)e * N + n] = 0;
        for (int x = 0; x < E; ++x) gain[(size_t)x * N + n] -= qq(x, e);
    }
    bool holds(int r, int e) const {
        return std::find(slots[r].begin(), slots[r].end(), e) != slots[r].end();
    }
    double rank_load(int r) const {
        std::vector<int32_t> ids = slots[r];
        std::sort(ids.begin(), ids.end());
        double l = 0.0;
        for (int e : ids) l += pl[(size_t)e * G + r];
        return l;
    }
    int single_node(int e) const {  // the node of a single expert, else -1
        int n1 = -1;
        for (int n = 0; n < N; ++n)
            if (on[(size_t)e * N + n]) {
                if (n1 >= 0) return -1;
                n1 = n;
            }
        return n1 >= 0 && pieces[(size_t)e * N + n1] == 1 ? n1 : -1;
    }

    bool place_work(const std::vector<int32_t>& order);
    void local_search();
    void pack_node(int n);
    void repair_node(int n);
    void repair_global();
    void coactivation_replicas();
};

struct Pick {
    int node = -1;
    bool fits = false, room = false;
    int64_t gain = 0;
    double spare = 0.0;
};

bool Planner::place_work(const std::vector<int32_t>& order) {
    for (int e : order) {
        double rem = (double)w[e];
        bool placed = false;
        int last = -1;
        while (!placed || rem > 0.0) {
            Pick best;
            int64_t slots_now = node_slots;
            for (int pass = 0; pass < 2; ++pass) {
                const int64_t lim_slots = pass == 0 ? node_slots : all_slots;
                Pick p;
                for (int n = 0; n < N; ++n) {
                    if (on[(size_t)e * N + n] || used[n] >= lim_slots) continue;
                    const int64_t lim = std::min<int64_t>(lim_slots - used[n], g);
                    Pick c;
                    c.node = n;
                    c.spare = node_cap - work[n];
                    c.fits = rem <= c.spare && need(rem) <= lim;
                    c.room = c.spare > 0.0;
                    c.gain = gain[(size_t)e * N + n];
                    const bool better =
                        p.node < 0 || c.fits > p.fits ||
                        (c.fits == p.fits &&
                         (c.room > p.room ||
                          (c.room == p.room &&
                           (c.spare > p.spare || (c.spare == p.spare && c.gain > p.gain)))));
                    if (better) p = c;
                }
                if (p.node >= 0 && (best.node < 0 || (p.fits && !best.fits))) {
                    best = p;
                    slots_now = lim_slots;
                }
                if (best.node >= 0 && best.fits) break;
            }
            if (best.node < 0) {
                if (!placed) return false;  // no slot left for this expert
                share[(size_t)e * N + last] += rem;
                work[last] += rem;
                rem = 0.0;
                break;
            }
            const int n = best.node;
            const int64_t lim = std::min<int64_t>(slots_now - used[n], g);
            double take = rem;
            if (!best.fits) {
                take = std::min(take, best.spare);
                take = std::min(take, (double)lim * cap);
                if (!(take > 0.0)) take = rem;
            }
            const int64_t k = std::min(need(take), lim);
            join(e, n);
            share[(size_t)e * N + n] = take;
            pieces[(size_t)e * N + n] = k;
            used[n] += k;
            work[n] += take;
            rem -= take;
            placed = true;
            last = n;
        }
    }
    return true;
}

void Planner::local_search() {
    std::vector<int> sn(E);  // node of each single expert, -1 otherwise
    for (int e = 0; e < E; ++e) sn[e] = single_node(e);
    for (int sweep = 0; sweep < 64; ++sweep) {
        bool changed = false;
        for (int a = 0; a < E; ++a) {
            const int na = sn[a];
            if (na < 0) continue;
            const double wa = (double)w[a];
            const int64_t ga = gain[(size_t)a * N + na];
            int64_t best = 0;
            int to = -1, partner = -1;
            for (int m = 0; m < N; ++m) {
                if (m == na || used[m] >= node_slots) continue;
                const double nw = work[m] + wa;
                if (!(nw <= node_cap || nw <= work[m])) continue;
                const int64_t d = gain[(size_t)a * N + m] - ga;
                if (d > best) {
                    best = d;
                    to = m;
                }
            }
            for (int b = 0; b < E; ++b) {
                const int nb = sn[b];
                if (b == a || nb < 0 || nb == na) continue;
                const double wb = (double)w[b];
                const double wna = work[na] - wa + wb, wnb = work[nb] - wb + wa;
                if (!(wna <= node_cap || wna <= work[na])) continue;
                if (!(wnb <= node_cap || wnb <= work[nb])) continue;
                // gains before the swap; b's own term q_ab is removed twice
                const int64_t d = gain[(size_t)a * N + nb] - ga + gain[(size_t)b * N + na] -
                                  gain[(size_t)b * N + nb] - 2 * qq(a, b);
                if (d > best) {
                    best = d;
                    to = -1;
                    partner = b;
                }
            }
            if (to >= 0) {
                leave(a, na);
                join(a, to);
                share[(size_t)a * N + to] = share[(size_t)a * N + na];
                share[(size_t)a * N + na] = 0.0;
                pieces[(size_t)a * N + to] = 1;
                pieces[(size_t)a * N + na] = 0;
                used[na] -= 1;
                used[to] += 1;
                work[na] = work[na] - wa;
                work[to] = work[to] + wa;
                sn[a] = to;
                changed = true;
            } else if (partner >= 0) {
                const int b = partner, nb = sn[b];
                const double wb = (double)w[b];
                leave(a, na);
                leave(b, nb);
                join(a, nb);
                join(b, na);
                share[(size_t)a * N + nb] = share[(size_t)a * N + na];
                share[(size_t)a * N + na] = 0.0;
                share[(size_t)b * N + na] = share[(size_t)b * N + nb];
                share[(size_t)b * N + nb] = 0.0;
                pieces[(size_t)a * N + nb] = 1;
                pieces[(size_t)a * N + na] = 0;
                pieces[(size_t)b * N + na] = 1;
                pieces[(size_t)b * N + nb] = 0;
                work[na] = work[na] - wa + wb;
                work[nb] = work[nb] - wb + wa;
                sn[a] = nb;
                sn[b] = na;
                changed = true;
            }
        }
        if (!changed) break;
    }
}

void Planner::pack_node(int n) {
    struct Piece {
        double load;
        int e, c;
    };
    std::vector<Piece> items;
    for (int e = 0; e < E; ++e) {
        if (!on[(size_t)e * N + n]) continue;
        const int64_t k = pieces[(size_t)e * N + n];
        for (int c = 0; c < k; ++c) items.push_back({share[(size_t)e * N + n] / (double)k, e, c});
    }
    std::stable_sort(items.begin(), items.end(), [](const Piece& a, const Piece& b) {
        if (a.load != b.load) return a.load > b.load;
        if (a.e != b.e) return a.e < b.e;
        return a.c < b.c;
    });
    const int ni = (int)items.size();
    const int lim = std::min(S, (ni + g - 1) / g);
    std::vector<double> load(g, 0.0);
    bool stuck = false;
    for (const Piece& it : items) {
        int b = -1;
        for (int i = 0; i < g; ++i) {
            const int r = n * g + i;
            if ((int)slots[r].size() >= lim || holds(r, it.e)) continue;
            if (b < 0 || load[i] < load[b] ||
                (load[i] == load[b] && slots[r].size() < slots[n * g + b].size()))
                b = i;
        }
        if (b < 0) {
            stuck = true;
            break;
        }
        const int r = n * g + b;
        slots[r].push_back(it.e);
        load[b] += it.load;
        pl[(size_t)it.e * G + r] += it.load;
    }
    if (!stuck) return;
    // round-robin: experts by decreasing piece count (ties smaller e), the
    // node's p-th piece on rank p mod g
    for (int i = 0; i < g; ++i) {
        const int r = n * g + i;
        slots[r].clear();
        for (int e = 0; e < E; ++e) pl[(size_t)e * G + r] = 0.0;
    }
    std::vector<int> ex;
    for (int e = 0; e < E; ++e)
        if (on[(size_t)e * N + n]) ex.push_back(e);
    std::stable_sort(ex.begin(), ex.end(), [&](int a, int b) {
        return pieces[(size_t)a * N + n] > pieces[(size_t)b * N + n];
    });
    int p = 0;
    for (int e : ex) {
        const int64_t k = pieces[(size_t)e * N + n];
        for (int64_t c = 0; c < k; ++c, ++p) {
            const int r = n * g + p % g;
            slots[r].push_back(e);
            pl[(size_t)e * G + r] += share[(size_t)e * N + n] / (double)k;
        }
    }
}

void Planner::repair_node(int n) {
    const int base = n * g;
    for (int64_t moves = 0; moves < 4 * (int64_t)g * g * S; ++moves) {
        int h = -1;
        double hl = 0.0;
        for (int i = 0; i < g; ++i) {
            const double l = rank_load(base + i);
            if (h < 0 || l > hl) {
                h = i;
                hl = l;
            }
        }
        if (!(hl > cap)) return;

        // breadth-first search for an augmenting path h -> ... -> target
        std::vector<int> queue{h}, parent(g, -1), via(g, -1);
        std::vector<uint8_t> seen(g, 0);
        seen[h] = 1;
        int target = -1;
        for (size_t qh = 0; qh < queue.size() && target < 0; ++qh) {
            const int a = queue[qh], ra = base + a;
            std::vector<int32_t> ids = slots[ra];
            std::sort(ids.begin(), ids.end());
            for (size_t t = 0; t < ids.size() && target < 0; ++t) {
                const int e = ids[t];
                if (!(pl[(size_t)e * G + ra] > 0.0)) continue;
                for (int b = 0; b < g && target < 0; ++b) {
                    const int rb = base + b;
                    if (seen[b]) continue;
                    if (!holds(rb, e) && (int)slots[rb].size() >= S) continue;
                    seen[b] = 1;
                    parent[b] = a;
                    via[b] = e;
                    queue.push_back(b);
                    if (rank_load(rb) < cap) target = b;
                }
            }
        }
        if (target >= 0) {
            double mv = std::min(hl - cap, cap - rank_load(base + target));
            for (int b = target; b != h; b = parent[b])
                mv = std::min(mv, pl[(size_t)via[b] * G + base + parent[b]]);
            if (!(mv > cap * 1e-12)) return;
            for (int b = target; b != h; b = parent[b]) {
                const int e = via[b], ra = base + parent[b], rb = base + b;
                if (!holds(rb, e)) slots[rb].push_back(e);
                pl[(size_t)e * G + ra] -= mv;
                pl[(size_t)e * G + rb] += mv;
            }
            continue;
        }

        // slot swap through h's free slot
        const int rh = base + h;
        if ((int)slots[rh].size() >= S) return;
        int eh = -1;
        for (int x : slots[rh])
            if (eh < 0 || pl[(size_t)x * G + rh] > pl[(size_t)eh * G + rh] ||
                (pl[(size_t)x * G + rh] == pl[(size_t)eh * G + rh] && x < eh))
                eh = x;
        const double weh = pl[(size_t)eh * G + rh];
        int bu = -1, bx = -1;
        double bul = 0.0;
        for (int u = 0; u < g; ++u) {
            const int ru = base + u;
            const double lu = rank_load(ru);
            if (u == h || !(lu < cap) || (int)slots[ru].size() < S || holds(ru, eh)) continue;
            int x = -1;
            for (int y : slots[ru]) {
                if (holds(rh, y) || !(pl[(size_t)y * G + ru] < weh)) continue;
                if (x < 0 || pl[(size_t)y * G + ru] < pl[(size_t)x * G + ru] ||
                    (pl[(size_t)y * G + ru] == pl[(size_t)x * G + ru] && y < x))
                    x = y;
            }
            if (x < 0) continue;
            if (bu < 0 || lu < bul) {
                bu = u;
                bx = x;
                bul = lu;
            }
        }
        if (bu < 0) return;
        const int ru = base + bu;
        const double wx = pl[(size_t)bx * G + ru];
        double mv = hl - cap + wx;
        mv = std::min(mv, cap - bul + wx);
        mv = std::min(mv, weh);
        if (!(mv > wx)) return;
        slots[ru].erase(std::find(slots[ru].begin(), slots[ru].end(), bx));
        slots[rh].push_back(bx);
        pl[(size_t)bx * G + ru] = 0.0;
        pl[(size_t)bx * G + rh] += wx;
        slots[ru].push_back(eh);
        pl[(size_t)eh * G + rh] -= mv;
        pl[(size_t)eh * G + ru] += mv;
    }
}

void Planner::repair_global() {
    std::vector<double> load(G);
    for (int r = 0; r < G; ++r) load[r] = rank_load(r);
    std::vector<int> queue, parent(G, -1), via(G, -1);
    std::vector<uint8_t> seen(G, 0);
    for (int64_t moves = 0; moves < 4 * (int64_t)G * S; ++moves) {
        int h = -1;
        double hl = 0.0;
        for (int r = 0; r < G; ++r)
            if (h < 0 || load[r] > hl) {
                h = r;
                hl = load[r];
            }
        if (!(hl > cap)) return;

        // held replicas first; new replicas in free slots only if that fails
        int target = -1;
        for (int phase = 0; phase < 2 && target < 0; ++phase) {
            queue.assign(1, h);
            std::fill(seen.begin(), seen.end(), 0);
            seen[h] = 1;
            for (size_t qh = 0; qh < queue.size() && target < 0; ++qh) {
                const int a = queue[qh];
                std::vector<int32_t> ids = slots[a];
                std::sort(ids.begin(), ids.end());
                for (size_t t = 0; t < ids.size() && target < 0; ++t) {
                    const int e = ids[t];
                    if (!(pl[(size_t)e * G + a] > 0.0)) continue;
                    for (int b = 0; b < G && target < 0; ++b) {
                        if (seen[b]) continue;
                        if (!holds(b, e) && (phase == 0 || (int)slots[b].size() >= S)) continue;
                        seen[b] = 1;
                        parent[b] = a;
                        via[b] = e;
                        queue.push_back(b);
                        if (cap - load[b] > cap * 1e-12) target = b;
                    }
                }
            }
        }
        if (target < 0) return;
        double mv = std::min(hl - cap, cap - load[target]);
        for (int b = target; b != h; b = parent[b])
            mv = std::min(mv, pl[(size_t)via[b] * G + parent[b]]);
        if (!(mv > cap * 1e-12)) return;
        for (int b = target; b != h; b = parent[b]) {
            const int e = via[b], a = parent[b], nb = b / g;
            if (!holds(b, e)) {
                slots[b].push_back(e);
                if (!on[(size_t)e * N + nb]) join(e, nb);
                used[nb] += 1;
            }
            pl[(size_t)e * G + a] -= mv;
            pl[(size_t)e * G + b] += mv;
        }
        for (int b = target; b != h; b = parent[b]) load[b] = rank_load(b);
        load[h] = rank_load(h);
    }
}

void Planner::coactivation_replicas() {
    for (;;) {
        int be = -1, bn = -1;
        int64_t bg = 0;
        for (int e = 0; e < E; ++e)
            for (int n = 0; n < N; ++n) {
                if (on[(size_t)e * N + n] || used[n] >= all_slots) continue;
                const int64_t gn = gain[(size_t)e * N + n];
                if (gn <= 0) continue;
                if (be < 0 || gn > bg || (gn == bg && w[e] > w[be])) {
                    be = e;
                    bn = n;
                    bg = gn;
                }
            }
        if (be < 0) return;
        int b = -1;
        for (int i = 0; i < g; ++i) {
            const int r = bn * g + i;
            if ((int)slots[r].size() >= S) continue;
            if (b < 0 || slots[r].size() < slots[bn * g + b].size()) b = i;
        }
        slots[bn * g + b].push_back(be);
        join(be, bn);
        used[bn] += 1;
    }
}

// One run of the steps with the node work bound of step 1 and its local
// search at node_frac * g * cap. Arguments are checked by the caller.
cobalt_status plan_once(int32_t N, int32_t gpn, int32_t E, int32_t S, const float* coact_ema,
                        const float* count_ema, float eps, double node_frac, int32_t* slot_table,
                        int32_t* owner, float* plan, double* objective, int32_t* feasible) {
    const int G = N * gpn;
    Planner P;
    P.N = N;
    P.g = gpn;
    P.G = G;
    P.E = E;
    P.S = S;
    P.w = count_ema;
    P.q.assign((size_t)E * E, 0);
    for (int i = 0; i < E; ++i)
        for (int j = i + 1; j < E; ++j)
            P.q[(size_t)i * E + j] = (int64_t)std::llrint(256.0 * (double)coact_ema[(size_t)i * E + j]);
    P.gain.assign((size_t)E * N, 0);
    P.on.assign((size_t)E * N, 0);
    P.share.assign((size_t)E * N, 0.0);
    P.pieces.assign((size_t)E * N, 0);
    P.used.assign(N, 0);
    P.work.assign(N, 0.0);
    P.slots.assign(G, {});
    P.pl.assign((size_t)E * G, 0.0);

    double W = 0.0;
    for (int e = 0; e < E; ++e) W += (double)count_ema[e];
    P.cap = (1.0 + (double)eps) * W / (double)G;
    P.node_cap = (double)gpn * P.cap * node_frac;
    P.all_slots = (int64_t)gpn * S;
    int64_t total_need = 0;
    for (int e = 0; e < E; ++e) total_need += P.need((double)count_ema[e]);
    const int64_t reserve =
        std::min<int64_t>(gpn, (int64_t)G * S > total_need ? ((int64_t)G * S - total_need) / N : 0);
    P.node_slots = P.all_slots - reserve;

    std::vector<int32_t> order(E);
    for (int e = 0; e < E; ++e) order[e] = e;
    std::stable_sort(order.begin(), order.end(),
                     [&](int a, int b) { return count_ema[a] > count_ema[b]; });

    if (!P.place_work(order)) return COBALT_EDATA;
    P.local_search();
    for (int n = 0; n < N; ++n) {
        P.pack_node(n);
        P.repair_node(n);
        P.used[n] = 0;
        for (int i = 0; i < gpn; ++i) P.used[n] += (int64_t)P.slots[n * gpn + i].size();
    }
    P.repair_global();
    P.coactivation_replicas();

    for (int r = 0; r < G; ++r)
        for (int k = 0; k < S; ++k)
            slot_table[(size_t)r * S + k] = k < (int)P.slots[r].size() ? P.slots[r][k] : -1;
    for (int e = 0; e < E; ++e) {
        int o = -1;
        for (int r = 0; r < G; ++r)
            if (P.holds(r, e) && (o < 0 || P.pl[(size_t)e * G + r] > P.pl[(size_t)e * G + o])) o = r;
        owner[e] = o;
    }
    if (plan)
        for (size_t i = 0; i < (size_t)E * G; ++i) plan[i] = (float)P.pl[i];
    if (objective) {
        int64_t obj = 0;
        for (int n = 0; n < N; ++n)
            for (int i = 0; i < E; ++i) {
                if (!P.on[(size_t)i * N + n]) continue;
                for (int j = i + 1; j < E; ++j)
                    if (P.on[(size_t)j * N + n]) obj += P.q[(size_t)i * E + j];
            }
        *objective = (double)obj / 256.0;
    }
    if (feasible) {
        int ok = 1;
        for (int r = 0; r < G; ++r)
            if (P.rank_load(r) > P.cap * (1.0 + 1e-9)) ok = 0;
        *feasible = ok;
    }
    return COBALT_OK;
}

}  // namespace
}  // namespace cobalt

using namespace cobalt;

extern "C" cobalt_status cobalt_plan_layout(int32_t N, int32_t gpn, int32_t E, int32_t S,
                                            const float* coact_ema, const float* count_ema,
                                            float eps, int32_t* slot_table, int32_t* owner,
                                            float* plan, double* objective,
                                            int32_t* feasible) {
    if (!coact_ema || !count_ema || !slot_table || !owner) return COBALT_EINVAL;
    if (N < 1 || N > kMaxN || gpn < 1 || gpn > kMaxGpn || E < 1 || E > kMaxE || S < 1)
        return COBALT_EINVAL;
    if (!(eps >= 0.0f) || std::isinf(eps)) return COBALT_EINVAL;
    const int G = N * gpn;
    if ((int64_t)G * S < E) return COBALT_EINVAL;
    for (int e = 0; e < E; ++e)
        if (!(count_ema[e] >= 0.0f) || std::isinf(count_ema[e])) return COBALT_EDATA;
    for (int i = 0; i < E; ++i)
        for (int j = i + 1; j < E; ++j) {
            const float c = coact_ema[(size_t)i * E + j];
            // q <= 2^36: the objective, at most kMaxN nodes x E(E-1)/2 < 2^23
            // pairs of them, stays below 2^63
            if (!(c >= 0.0f) || !(c <= 268435456.0f)) return COBALT_EDATA;  // 2^28
        }

    int32_t ok = 0;
    cobalt_status st = plan_once(N, gpn, E, S, coact_ema, count_ema, eps, 1.0, slot_table, owner,
                                 plan, objective, &ok);
    if (st != COBALT_OK || ok) {
        if (st == COBALT_OK && feasible) *feasible = ok;
        return st;
    }
    // above the cap: retry with slack left on every node by steps 1 and 1b
    static const double retry[3] = {0.98, 0.95, 0.90};
    std::vector<int32_t> t2((size_t)G * S), o2(E);
    std::vector<float> p2((size_t)E * G);
    for (int k = 0; k < 3 && !ok; ++k) {
        double obj2 = 0.0;
        int32_t ok2 = 0;
        if (plan_once(N, gpn, E, S, coact_ema, count_ema, eps, retry[k], t2.data(), o2.data(),
                      p2.data(), &obj2, &ok2) != COBALT_OK ||
            !ok2)
            continue;
        std::copy(t2.begin(), t2.end(), slot_table);
        std::copy(o2.begin(), o2.end(), owner);
        if (plan) std::copy(p2.begin(), p2.end(), plan);
        if (objective) *objective = obj2;
        ok = 1;
    }
    if (feasible) *feasible = ok;
    return COBALT_OK;
}

