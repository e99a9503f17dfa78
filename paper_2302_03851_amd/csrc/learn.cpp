// Learning the FSM batching policy (Section 2.3 of ED-Batch): tabular
// Q-learning with N-step bootstrapping over the batching loop of Algorithm 1,
// with the reward of Eq. 1.  Host only; the result is a policy table in the
// format edb_schedule reads.
#include <algorithm>
#include <map>
#include <new>
#include <string>

#include "edb_internal.h"

struct edb_learned {
    int32_t T = 0;
    std::vector<int32_t> table;
    std::vector<int32_t> q_keys;
    std::vector<double> q;
    int32_t n_q_states = 0;
    edb_learn_stats stats{};
};

namespace {

using edb::fail;
using Key = std::vector<int32_t>;
using QTable = std::map<Key, std::vector<double>>;

// SplitMix64 (Steele, Lea and Flood 2014): a Weyl sequence through the
// variant-13 64-bit finalizer; draw k of a seed is stateless.
uint64_t splitmix64(uint64_t seed, uint64_t k) {
    uint64_t z = seed + (k + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

int32_t majority(const std::vector<int64_t>& counts) {
    int32_t best = -1;
    for (int32_t t = 0; t < (int32_t)counts.size(); ++t)
        if (counts[t] > 0 && (best < 0 || counts[t] > counts[best])) best = t;
    return best;
}

// State key E(G) of Section 2.3 and the actions it offers (frontier types in
// key order; E_max's last entry repeats the majority type).
void state_of(const std::vector<int64_t>& counts, int32_t enc, Key& key, int32_t& n_actions) {
    key.clear();
    for (int32_t t = 0; t < (int32_t)counts.size(); ++t)
        if (counts[t] > 0) key.push_back(t);
    if (enc == EDB_ENC_SORT)
        std::stable_sort(key.begin(), key.end(), [&](int32_t a, int32_t b) { return counts[a] > counts[b]; });
    n_actions = (int32_t)key.size();
    if (enc == EDB_ENC_MAX) key.push_back(majority(counts));
}

double qval(const QTable& Q, const Key& key, int32_t a) {
    auto it = Q.find(key);
    return it == Q.end() ? 0.0 : it->second[a];
}

int32_t greedy(const QTable& Q, const Key& key, int32_t n_actions) {
    auto it = Q.find(key);
    int32_t best = key[0];
    if (it == Q.end()) return best;
    for (int32_t i = 1; i < n_actions; ++i)
        if (it->second[key[i]] > it->second[best]) best = key[i];
    return best;
}

int32_t actions_of(const Key& key, int32_t enc) {
    return enc == EDB_ENC_MAX ? (int32_t)key.size() - 1 : (int32_t)key.size();
}

// G_t of Algorithm 1: the frontier per type plus the sub-frontier counts of
// each type's induced subgraph.
struct Episode {
    const edb_graph& g;
    std::vector<int32_t> pending, same_pending;
    std::vector<std::vector<int32_t>> ready;
    std::vector<int64_t> counts, subf;
    int64_t left;

    explicit Episode(const edb_graph& graph) : g(graph), pending(graph.pending), ready(graph.T),
                                               counts(graph.T, 0), left(graph.V) {
        for (int32_t v = 0; v < g.V; ++v) if (pending[v] == 0) ready[g.op_type[v]].push_back(v);
        for (int32_t t = 0; t < g.T; ++t) counts[t] = (int64_t)ready[t].size();
        edb::same_type_frontier(g, same_pending, subf);
    }
    // Eq. 1 for action a before it executes
    double reward(int32_t a, double alpha) const {
        return -1.0 + alpha * ((double)counts[a] / (double)subf[a]);
    }
    void execute(int32_t a) {
        std::vector<int32_t> batch;
        batch.swap(ready[a]);
        for (int32_t v : batch) {
            edb::same_type_executed(g, v, same_pending, subf);
            for (int32_t i = g.cons_ptr[v]; i < g.cons_ptr[v + 1]; ++i) {
                const int32_t p = g.cons[i];
                if (--pending[p] == 0) ready[g.op_type[p]].push_back(p);
            }
        }
        left -= (int64_t)batch.size();
        for (int32_t t = 0; t < g.T; ++t) counts[t] = (int64_t)ready[t].size();
    }
};

void flatten(const QTable& Q, int32_t enc, std::vector<int32_t>& flat) {
    flat.assign(1, (int32_t)Q.size());
    for (const auto& kv : Q) {
        flat.push_back((int32_t)kv.first.size());
        flat.insert(flat.end(), kv.first.begin(), kv.first.end());
        flat.push_back(greedy(Q, kv.first, actions_of(kv.first, enc)));
    }
}

}  // namespace

extern "C" void edb_learn_defaults(edb_learn_params* p) {
    if (!p) return;
    p->encoding = EDB_ENC_SORT;
    p->trials = 1000;
    p->check_every = 50;
    p->n_step = 4;
    p->alpha = 0.5;
    p->epsilon = 0.1;
    p->lr = 0.2;
    p->gamma = 1.0;
    p->seed = 0;
}

extern "C" edb_status edb_learn_policy(const edb_graph_t* g, const edb_learn_params* p, edb_learned_t** out) {
    if (!out) return fail(EDB_ERR_INVALID, "edb_learn_policy: out is NULL");
    *out = nullptr;
    if (!g || !p) return fail(EDB_ERR_INVALID, "edb_learn_policy: NULL graph or parameters");
    if (p->encoding < EDB_ENC_SORT || p->encoding > EDB_ENC_MAX)
        return fail(EDB_ERR_INVALID, "edb_learn_policy: unknown state encoding");
    if (p->trials < 1 || p->check_every < 1 || p->n_step < 1)
        return fail(EDB_ERR_INVALID, "edb_learn_policy: trials, check_every and n_step must be >= 1");
    if (!(p->alpha > 0.0) || !(p->epsilon >= 0.0 && p->epsilon <= 1.0) || !(p->lr > 0.0 && p->lr <= 1.0) ||
        !(p->gamma >= 0.0 && p->gamma <= 1.0))
        return fail(EDB_ERR_INVALID, "edb_learn_policy: alpha, epsilon, lr or gamma out of range");

    edb_learned* L = new (std::nothrow) edb_learned;
    if (!L) return fail(EDB_ERR_OOM, "edb_learn_policy: out of host memory");
    try {
        const int32_t enc = p->encoding, N = p->n_step, T = g->T;
        const int64_t lb = edb::lower_bound(*g);
        QTable Q;
        uint64_t c = 0;  // training step counter over all trials
        std::vector<int32_t> best_table, flat;
        int32_t best_nb = -1, trial = 0;
        std::vector<Key> states;
        std::vector<int32_t> acts;
        std::vector<double> rews;
        Key key;

        // N-step target for step tau; T_end < 0 while the episode runs
        auto update = [&](int64_t tau, int64_t T_end) {
            double ret = 0.0, mult = 1.0;
            const int64_t stop = T_end < 0 ? tau + N : std::min<int64_t>(tau + N, T_end);
            for (int64_t i = tau; i < stop; ++i) {
                ret = ret + mult * rews[i];
                mult = mult * p->gamma;
            }
            if (T_end < 0 || tau + N < T_end) {
                const Key& nxt = states[tau + N];
                double m = qval(Q, nxt, nxt[0]);
                for (int32_t i = 1; i < actions_of(nxt, enc); ++i) m = std::max(m, qval(Q, nxt, nxt[i]));
                ret = ret + mult * m;
            }
            auto it = Q.find(states[tau]);
            if (it == Q.end()) it = Q.emplace(states[tau], std::vector<double>(T, 0.0)).first;
            double& q = it->second[acts[tau]];
            q = q + p->lr * (ret - q);
        };

        while (trial < p->trials) {
            ++trial;
            Episode ep(*g);
            states.clear();
            acts.clear();
            rews.clear();
            int64_t t = 0;
            int32_t na = 0;
            if (ep.left > 0) {
                state_of(ep.counts, enc, key, na);
                states.push_back(key);
            }
            while (ep.left > 0) {
                const Key& s = states[t];
                const int32_t n_act = actions_of(s, enc);
                int32_t a;
                const double u = (double)(splitmix64(p->seed, 2 * c) >> 11) * 0x1p-53;
                if (u < p->epsilon)
                    a = s[splitmix64(p->seed, 2 * c + 1) % (uint64_t)n_act];
                else
                    a = greedy(Q, s, n_act);
                ++c;
                const double r = ep.reward(a, p->alpha);
                ep.execute(a);
                acts.push_back(a);
                rews.push_back(r);
                ++t;
                if (ep.left > 0) {
                    state_of(ep.counts, enc, key, na);
                    states.push_back(key);
                    if (t - N >= 0) update(t - N, -1);
                } else {
                    for (int64_t tau = std::max<int64_t>(0, t - N); tau < t; ++tau) update(tau, t);
                }
            }
            if (trial % p->check_every == 0 || trial == p->trials) {
                flatten(Q, enc, flat);
                edb_policy pol{EDB_POLICY_TABLE, enc, flat.data(), (int64_t)flat.size()};
                edb_schedule_t* s = nullptr;
                edb_status st = edb_schedule(g, &pol, &s);
                if (st != EDB_OK) {
                    delete L;
                    return st;
                }
                const int32_t nb = (int32_t)s->batch_type.size();
                edb_schedule_free(s);
                if (best_nb < 0 || nb < best_nb) {
                    best_nb = nb;
                    best_table = flat;
                }
                if (best_nb <= lb) break;
            }
        }
        L->T = T;
        L->table = best_table;
        L->stats.trials = trial;
        L->stats.batches = best_nb;
        L->stats.lower_bound = lb;
        L->stats.n_states = best_table.empty() ? 0 : best_table[0];
        L->n_q_states = (int32_t)Q.size();
        for (const auto& kv : Q) {
            L->q_keys.push_back((int32_t)kv.first.size());
            L->q_keys.insert(L->q_keys.end(), kv.first.begin(), kv.first.end());
            L->q.insert(L->q.end(), kv.second.begin(), kv.second.end());
        }
    } catch (const std::bad_alloc&) {
        delete L;
        return fail(EDB_ERR_OOM, "edb_learn_policy: out of host memory");
    } catch (const std::exception& e) {
        delete L;
        return fail(EDB_ERR_INVALID, std::string("edb_learn_policy: internal error: ") + e.what());
    }
    edb::clear_error();
    *out = L;
    return EDB_OK;
}

extern "C" edb_status edb_learned_view(const edb_learned_t* l, const int32_t** table, int64_t* table_len,
                                       edb_learn_stats* stats) {
    if (!l) return fail(EDB_ERR_INVALID, "edb_learned_view: handle is NULL");
    if (table) *table = l->table.data();
    if (table_len) *table_len = (int64_t)l->table.size();
    if (stats) *stats = l->stats;
    return EDB_OK;
}

extern "C" edb_status edb_learned_q(const edb_learned_t* l, int32_t* n_states, const int32_t** keys,
                                    int64_t* keys_len, const double** q) {
    if (!l) return fail(EDB_ERR_INVALID, "edb_learned_q: handle is NULL");
    if (n_states) *n_states = l->n_q_states;
    if (keys) *keys = l->q_keys.data();
    if (keys_len) *keys_len = (int64_t)l->q_keys.size();
    if (q) *q = l->q.data();
    return EDB_OK;
}

extern "C" void edb_learned_free(edb_learned_t* l) { delete l; }
