// Per-step intra-node rebalancing (Section 3.2, Stage 2), host side.
//
// Within each node the replicas currently placed on the node's ranks are
// re-partitioned among those ranks to lower the highest rank load: the
// replicas are sorted by estimated workload (heaviest first) and each goes
// to the least-loaded rank of the node that still has a free slot and does
// not already hold a replica of the same expert (at most S slots per rank,
// no two replicas of one expert on a rank). Which replicas exist on a node
// is unchanged, so nothing crosses a node boundary. If the greedy pass finds
// no eligible rank for some replica, that node keeps its previous placement.
#include <algorithm>
#include <cmath>
#include <vector>

#include "internal.hpp"

using namespace cobalt;

extern "C" cobalt_status cobalt_intra_node_rebalance(int32_t N, int32_t gpn, int32_t E, int32_t S,
                                                     const int32_t* slot, const int32_t* owner_in,
                                                     const float* rload, int32_t* new_slot,
                                                     int32_t* new_owner, float* rank_load) {
    if (!slot || !rload || !new_slot) return COBALT_EINVAL;
    if (N < 1 || N > kMaxN || gpn < 1 || gpn > kMaxGpn || E < 1 || E > kMaxE || S < 1)
        return COBALT_EINVAL;
    const int32_t G = N * gpn;
    if (G > kMaxG) return COBALT_EUNSUPPORTED;

    // validate the table and find the owner replica of each expert
    std::vector<uint8_t> held((size_t)G * E, 0);
    std::vector<int32_t> owner(E, -1);
    for (int32_t r = 0; r < G; ++r)
        for (int32_t k = 0; k < S; ++k) {
            const int32_t e = slot[(size_t)r * S + k];
            if (e == -1) continue;
            if (e < 0 || e >= E || held[(size_t)r * E + e]) return COBALT_EDATA;
            held[(size_t)r * E + e] = 1;
            if (owner[e] < 0) owner[e] = r;
        }
    for (int32_t e = 0; e < E; ++e) {
        if (owner[e] < 0) return COBALT_EDATA;
        if (owner_in) {
            const int32_t o = owner_in[e];
            if (o < 0 || o >= G || !held[(size_t)o * E + e]) return COBALT_EDATA;
            owner[e] = o;
        }
    }

    // the load of every placed replica must be finite and non-negative
    for (int32_t r = 0; r < G; ++r)
        for (int32_t k = 0; k < S; ++k) {
            const int32_t e = slot[(size_t)r * S + k];
            if (e < 0) continue;
            const float l = rload[(size_t)e * G + r];
            if (!std::isfinite(l) || l < 0.f) return COBALT_EDATA;
        }

    std::vector<int32_t> out((size_t)G * S, -1);
    std::vector<int32_t> own = owner;
    std::vector<float> rl(G, 0.f);
    struct Rep {
        float load;
        int32_t e, r;
    };
    for (int32_t n = 0; n < N; ++n) {
        std::vector<Rep> reps;
        for (int32_t i = 0; i < gpn; ++i) {
            const int32_t r = n * gpn + i;
            for (int32_t k = 0; k < S; ++k) {
                const int32_t e = slot[(size_t)r * S + k];
                if (e >= 0) reps.push_back({rload[(size_t)e * G + r], e, r});
            }
        }
        std::stable_sort(reps.begin(), reps.end(), [](const Rep& a, const Rep& b) {
            if (a.load != b.load) return a.load > b.load;
            if (a.e != b.e) return a.e < b.e;
            return a.r < b.r;
        });
        std::vector<float> load(gpn, 0.f);
        std::vector<int32_t> used(gpn, 0);
        std::vector<uint8_t> has((size_t)gpn * E, 0);
        std::vector<int32_t> dest(reps.size(), -1);
        bool ok = true;
        for (size_t q = 0; q < reps.size() && ok; ++q) {
            int32_t best = -1;
            for (int32_t i = 0; i < gpn; ++i) {
                if (used[i] >= S || has[(size_t)i * E + reps[q].e]) continue;
                if (best < 0 || load[i] < load[best]) best = i;
            }
            if (best < 0) {
                ok = false;
                break;
            }
            dest[q] = best;
            load[best] += reps[q].load;
            has[(size_t)best * E + reps[q].e] = 1;
            ++used[best];
        }
        if (ok) {
            std::vector<int32_t> fill(gpn, 0);
            for (size_t q = 0; q < reps.size(); ++q) {
                const int32_t r = n * gpn + dest[q];
                out[(size_t)r * S + fill[dest[q]]++] = reps[q].e;
                if (owner[reps[q].e] == reps[q].r) own[reps[q].e] = r;
            }
            for (int32_t i = 0; i < gpn; ++i) rl[n * gpn + i] = load[i];
        } else {
            for (int32_t i = 0; i < gpn; ++i) {
                const int32_t r = n * gpn + i;
                float l = 0.f;
                for (int32_t k = 0; k < S; ++k) {
                    const int32_t e = slot[(size_t)r * S + k];
                    out[(size_t)r * S + k] = e;
                    if (e >= 0) l += rload[(size_t)e * G + r];
                }
                rl[r] = l;
            }
        }
    }
    std::copy(out.begin(), out.end(), new_slot);
    if (new_owner) std::copy(own.begin(), own.end(), new_owner);
    if (rank_load) std::copy(rl.begin(), rl.end(), rank_load);
    return COBALT_OK;
}
