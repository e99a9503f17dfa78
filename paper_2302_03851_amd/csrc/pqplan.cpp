// PQ-tree memory layout (Section 3.2 of ED-Batch, Algorithm 2 and Appendix B):
// an arena order in which the operands of as many batches as possible are
// contiguous and aligned with their rows.
//
// Variables are the node states plus one zero pad per absent entry of a
// positional operand list that has a present entry.  A batch's aligned
// operands are its rows (ascending id) and, per positional child p, the list
// of the rows' p-th children (or pads), kept when it has no repeated entry;
// a ragged child list only asks for adjacency.
//
//   construct  every operand set is reduced into a PQ tree (Booth and
//              Lueker's templates), batches last to first, in a batch the
//              child lists, the ragged set, then the rows; an operand whose
//              set cannot be made consecutive leaves the batch's aligned
//              group (the rows then follow the group's first operand and the
//              results scatter)
//   broadcast  the structure covering each operand of a group (P-node leaf
//              sets, pairs of neighbouring Q-node children) is read in row
//              positions, the union over the group is mapped onto every
//              operand and reduced; sweeps repeat until nothing changes
//   decide     matching structures give order relations (a direction parity
//              between Q-nodes, a child bijection between P-nodes) merged by
//              a union-find that keeps each node's order relative to its
//              parent; contradicting relations are dropped
//   leaf order depth-first, every node in the order its class root implies
// Nodes with two children count as Q-nodes in the last two steps (their two
// orders are each other's reversal).  The reduction checks every template
// before it restructures anything, so a failed set leaves the tree unchanged.
#include <algorithm>
#include <map>
#include <set>
#include <vector>

#include "edb_internal.h"

namespace {

enum { LEAF = 0, PNODE = 1, QNODE = 2 };
enum { EMPTY = 0, FULL = 1, PARTIAL = 2 };

struct PQTree {
    std::vector<int> kind, parent;
    std::vector<std::vector<int>> children;
    int root = -1;
    // scratch for one reduction
    std::vector<int> cnt, st, touched;

    explicit PQTree(int n) : kind(n, LEAF), parent(n, -1), children(n) {
        if (n >= 2) {
            std::vector<int> all(n);
            for (int i = 0; i < n; ++i) all[i] = i;
            root = add(PNODE, all);
        } else {
            root = n == 1 ? 0 : -1;
        }
    }
    int add(int k, const std::vector<int>& kids) {
        const int i = (int)kind.size();
        kind.push_back(k);
        parent.push_back(-1);
        children.push_back(kids);
        for (int c : kids) parent[c] = i;
        return i;
    }
    void set_children(int x, std::vector<int> kids) {
        for (int c : kids) parent[c] = x;
        children[x] = std::move(kids);
    }
    void replace(int old, int nw) {
        const int p = parent[old];
        parent[nw] = p;
        if (p < 0) root = nw;
        else
            for (int& c : children[p]) if (c == old) c = nw;
    }
    void leaves(int x, std::vector<int>& out) const {
        std::vector<int> stack{x};
        while (!stack.empty()) {
            const int y = stack.back();
            stack.pop_back();
            if (kind[y] == LEAF) { out.push_back(y); continue; }
            for (auto it = children[y].rbegin(); it != children[y].rend(); ++it) stack.push_back(*it);
        }
    }
    int order_kind(int x) const {
        return (kind[x] == QNODE || children[x].size() == 2) ? QNODE : PNODE;
    }

    // pertinent counts: cnt[y] = leaves of S under y (only for y touched)
    void count(const std::vector<int>& S) {
        if (cnt.size() < kind.size()) { cnt.resize(kind.size(), 0); st.resize(kind.size(), EMPTY); }
        for (int y : touched) { cnt[y] = 0; st[y] = EMPTY; }
        touched.clear();
        for (int s : S)
            for (int y = s; y >= 0; y = parent[y]) {
                if (cnt[y] == 0) touched.push_back(y);
                ++cnt[y];
            }
    }
    int pertinent_root(const std::vector<int>& S) {
        count(S);
        int x = S[0];
        while (cnt[x] != (int)S.size()) x = parent[x];
        return x;
    }
    int status(int x) {
        if (cnt[x] == 0) return st[x] = EMPTY;
        if (kind[x] == LEAF) return st[x] = FULL;
        bool all_full = true;
        for (int c : children[x]) all_full &= status(c) == FULL;
        return st[x] = all_full ? FULL : PARTIAL;
    }
    int stat(int c) const { return cnt[c] == 0 ? EMPTY : st[c]; }

    static bool q_pattern(const std::vector<int>& seq, bool at_root) {
        size_t i = 0, n = seq.size();
        while (i < n && seq[i] == EMPTY) ++i;
        if (i < n && seq[i] == PARTIAL) ++i;
        while (i < n && seq[i] == FULL) ++i;
        if (at_root) {
            if (i < n && seq[i] == PARTIAL) ++i;
            while (i < n && seq[i] == EMPTY) ++i;
        }
        return i == n;
    }
    std::vector<int> seq_of(int x) const {
        std::vector<int> s;
        for (int c : children[x]) s.push_back(stat(c));
        return s;
    }
    bool check(int x, bool at_root) {
        if (stat(x) != PARTIAL) return true;
        for (int c : children[x])
            if (stat(c) == PARTIAL && !check(c, false)) return false;
        const std::vector<int> seq = seq_of(x);
        const long np = std::count(seq.begin(), seq.end(), PARTIAL);
        if (kind[x] == PNODE) return np <= (at_root ? 2 : 1);
        if (at_root) return q_pattern(seq, true);
        std::vector<int> rev(seq.rbegin(), seq.rend());
        return q_pattern(seq, false) || q_pattern(rev, false);
    }
    bool implied(const std::vector<int>& S) {
        if (S.size() < 2) return true;
        const int x = pertinent_root(S);
        if (status(x) == FULL) return true;
        if (kind[x] != QNODE) return false;
        int first = -1, last = -1, nfull = 0;
        for (size_t i = 0; i < children[x].size(); ++i) {
            const int s = stat(children[x][i]);
            if (s == PARTIAL) return false;
            if (s == FULL) {
                if (first < 0) first = (int)i;
                last = (int)i;
                ++nfull;
            }
        }
        return nfull == last - first + 1;
    }
    std::vector<int> group(const std::vector<int>& kids) {
        if (kids.empty()) return {};
        if (kids.size() == 1) return {kids[0]};
        return {add(PNODE, kids)};
    }
    int apply(int x, bool at_root) {
        if (stat(x) != PARTIAL) return x;
        const std::vector<int> k0 = children[x];
        for (int c : k0)
            if (stat(c) == PARTIAL) apply(c, false);
        std::vector<int> kids = children[x], E, F, Pa;
        for (int c : kids) (stat(c) == EMPTY ? E : stat(c) == FULL ? F : Pa).push_back(c);
        if (kind[x] == PNODE && !at_root) {
            std::vector<int> out = group(E);
            const std::vector<int> gF = group(F);
            if (!Pa.empty()) out.insert(out.end(), children[Pa[0]].begin(), children[Pa[0]].end());
            out.insert(out.end(), gF.begin(), gF.end());
            kind[x] = QNODE;
            set_children(x, out);
            return x;
        }
        if (kind[x] == PNODE) {
            if (Pa.empty()) {
                if (F.size() >= 2) {
                    std::vector<int> out = E;
                    const std::vector<int> gF = group(F);
                    out.insert(out.end(), gF.begin(), gF.end());
                    set_children(x, out);
                }
                return x;
            }
            const int y = Pa[0];
            if (Pa.size() == 2) {
                const int y2 = Pa[1];
                const std::vector<int> gF = group(F);
                std::vector<int> out = children[y];
                out.insert(out.end(), gF.begin(), gF.end());
                out.insert(out.end(), children[y2].rbegin(), children[y2].rend());
                set_children(y, out);
            } else {
                std::vector<int> out = children[y];
                const std::vector<int> gF = group(F);
                out.insert(out.end(), gF.begin(), gF.end());
                set_children(y, out);
                if (children[y].size() == 2) kind[y] = PNODE;
            }
            if (!E.empty()) {
                std::vector<int> out = E;
                out.push_back(y);
                set_children(x, out);
                return x;
            }
            replace(x, y);
            return y;
        }
        if (!at_root) {
            if (!q_pattern(seq_of(x), false)) std::reverse(kids.begin(), kids.end());
            std::vector<int> out;
            for (int c : kids) {
                if (stat(c) == PARTIAL) out.insert(out.end(), children[c].begin(), children[c].end());
                else out.push_back(c);
            }
            set_children(x, out);
            return x;
        }
        std::vector<int> out;
        bool seen_full = false;
        for (int c : kids) {
            if (stat(c) == PARTIAL) {
                if (!seen_full) out.insert(out.end(), children[c].begin(), children[c].end());
                else out.insert(out.end(), children[c].rbegin(), children[c].rend());
                seen_full = true;
            } else {
                if (stat(c) == FULL) seen_full = true;
                out.push_back(c);
            }
        }
        set_children(x, out);
        return x;
    }
    // returns ok; *changed set when the tree was restructured
    bool reduce(const std::vector<int>& S, bool* changed) {
        *changed = false;
        if (S.size() < 2 || implied(S)) return true;
        const int x = pertinent_root(S);
        status(x);
        if (!check(x, true)) return false;
        const int top = apply(x, true);
        if (kind[top] == QNODE && children[top].size() == 2) kind[top] = PNODE;
        *changed = true;
        return true;
    }
};

// (kind, node, children) per structure element, depth-first pre-order
struct Elem {
    int kind, node;
    std::vector<int> kids;
};

void structure(PQTree& t, const std::vector<int>& o, std::vector<Elem>& out) {
    out.clear();
    const int r = t.pertinent_root(o);
    std::vector<int> lv;
    t.leaves(r, lv);
    std::vector<int> stack;
    auto visit = [&](int x) {
        stack.assign(1, x);
        while (!stack.empty()) {
            const int y = stack.back();
            stack.pop_back();
            if (t.kind[y] == LEAF) continue;
            out.push_back({t.order_kind(y), y, t.children[y]});
            for (auto it = t.children[y].rbegin(); it != t.children[y].rend(); ++it) stack.push_back(*it);
        }
    };
    if (lv.size() == o.size()) {   // the leaves of r hold o and are as many: exactly o
        visit(r);
        return;
    }
    const std::set<int> A(o.begin(), o.end());
    std::vector<int> kids;
    for (int c : t.children[r]) {
        std::vector<int> cl;
        t.leaves(c, cl);
        bool inside = true;
        for (int l : cl) inside &= A.count(l) > 0;
        if (inside) kids.push_back(c);
    }
    out.push_back({QNODE, r, kids});
    for (int c : kids) visit(c);
}

using PosSet = std::vector<int>;   // sorted positions

std::vector<PosSet> child_positions(PQTree& t, const std::vector<int>& kids, const std::map<int, int>& pos) {
    std::vector<PosSet> sets;
    for (int c : kids) {
        std::vector<int> cl;
        t.leaves(c, cl);
        PosSet s;
        for (int l : cl) s.push_back(pos.at(l));
        std::sort(s.begin(), s.end());
        sets.push_back(s);
    }
    return sets;
}

std::map<int, int> positions(const std::vector<int>& o) {
    std::map<int, int> pos;
    for (size_t i = 0; i < o.size(); ++i) pos[o[i]] = (int)i;
    return pos;
}

void parse_constraints(PQTree& t, const std::vector<const std::vector<int>*>& ops,
                       std::vector<std::vector<int>>& out) {
    std::vector<PosSet> uniform;
    std::set<PosSet> seen;
    std::vector<Elem> el;
    for (const std::vector<int>* o : ops) {
        structure(t, *o, el);
        const std::map<int, int> pos = positions(*o);
        for (const Elem& e : el) {
            const std::vector<PosSet> sets = child_positions(t, e.kids, pos);
            std::vector<PosSet> cons;
            if (e.kind == PNODE) {
                PosSet all;
                for (const PosSet& s : sets) all.insert(all.end(), s.begin(), s.end());
                std::sort(all.begin(), all.end());
                cons.push_back(all);
            } else {
                for (size_t i = 0; i + 1 < sets.size(); ++i) {
                    PosSet u = sets[i];
                    u.insert(u.end(), sets[i + 1].begin(), sets[i + 1].end());
                    std::sort(u.begin(), u.end());
                    cons.push_back(u);
                }
            }
            for (PosSet& c : cons)
                if (seen.insert(c).second) uniform.push_back(c);
        }
    }
    out.clear();
    for (const std::vector<int>* o : ops)
        for (const PosSet& c : uniform) {
            std::vector<int> vars;
            for (int i : c) vars.push_back((*o)[i]);
            out.push_back(vars);
        }
}

struct UnionFind {
    const PQTree& t;
    std::map<int, int> up;
    std::map<int, int> par;                  // Q: parity relative to up
    std::map<int, std::map<int, int>> sig;   // P: parent's child -> own child
    explicit UnionFind(const PQTree& tree) : t(tree) {}
    int upof(int x) const {
        auto it = up.find(x);
        return it == up.end() ? x : it->second;
    }
    int find_q(int x, int* parity) const {
        int p = 0;
        while (upof(x) != x) {
            p ^= par.at(x);
            x = up.at(x);
        }
        *parity = p;
        return x;
    }
    int find_p(int x, std::map<int, int>& total) const {
        total.clear();
        for (int c : t.children[x]) total[c] = c;
        while (upof(x) != x) {
            const std::map<int, int>& s = sig.at(x);
            std::map<int, int> nt;
            for (const auto& kv : s) nt[kv.first] = total.at(kv.second);
            total.swap(nt);
            x = up.at(x);
        }
        return x;
    }
    bool union_q(int a, int b, int rel) {
        int pa, pb;
        const int ra = find_q(a, &pa), rb = find_q(b, &pb);
        if (ra == rb) return (pa ^ pb) == rel;
        up[ra] = rb;
        par[ra] = pa ^ pb ^ rel;
        return true;
    }
    bool union_p(int a, int b, const std::map<int, int>& f) {
        std::map<int, int> Ta, Tb;
        const int ra = find_p(a, Ta), rb = find_p(b, Tb);
        if (ra == rb) {
            for (const auto& kv : Ta)
                if (f.at(kv.second) != Tb.at(kv.first)) return false;
            return true;
        }
        std::map<int, int> finv, Tainv;
        for (const auto& kv : f) finv[kv.second] = kv.first;
        for (const auto& kv : Ta) Tainv[kv.second] = kv.first;
        std::map<int, int> s;
        for (const auto& kv : Tb) s[kv.first] = Tainv.at(finv.at(kv.second));
        up[ra] = rb;
        sig[ra] = s;
        return true;
    }
};

struct Relation {
    int kind, x, y, parity;
    std::map<int, int> f;
};

bool relations(PQTree& t, const std::vector<const std::vector<int>*>& ops, std::vector<Relation>& rels) {
    rels.clear();
    std::vector<Elem> s0, sj;
    structure(t, *ops[0], s0);
    const std::map<int, int> p0 = positions(*ops[0]);
    std::vector<std::vector<PosSet>> key0;
    for (const Elem& e : s0) key0.push_back(child_positions(t, e.kids, p0));
    for (size_t j = 1; j < ops.size(); ++j) {
        structure(t, *ops[j], sj);
        const std::map<int, int> pj = positions(*ops[j]);
        std::map<PosSet, std::pair<size_t, std::vector<PosSet>>> byset;
        for (size_t i = 0; i < sj.size(); ++i) {
            std::vector<PosSet> ks = child_positions(t, sj[i].kids, pj);
            PosSet u;
            for (const PosSet& s : ks) u.insert(u.end(), s.begin(), s.end());
            std::sort(u.begin(), u.end());
            byset[u] = {i, ks};
        }
        for (size_t e = 0; e < s0.size(); ++e) {
            const std::vector<PosSet>& ks = key0[e];
            PosSet u;
            for (const PosSet& s : ks) u.insert(u.end(), s.begin(), s.end());
            std::sort(u.begin(), u.end());
            auto it = byset.find(u);
            if (it == byset.end()) return false;
            const Elem& m = sj[it->second.first];
            const std::vector<PosSet>& yks = it->second.second;
            if (m.kind != s0[e].kind) return false;
            std::set<PosSet> a(ks.begin(), ks.end()), b(yks.begin(), yks.end());
            if (a != b || ks.size() != yks.size()) return false;
            if (s0[e].kind == QNODE) {
                std::vector<PosSet> rev(ks.rbegin(), ks.rend());
                if (yks == ks) rels.push_back({QNODE, s0[e].node, m.node, 0, {}});
                else if (yks == rev) rels.push_back({QNODE, s0[e].node, m.node, 1, {}});
                else return false;
            } else {
                std::map<PosSet, int> at;
                for (size_t i = 0; i < yks.size(); ++i) at[yks[i]] = m.kids[i];
                Relation r{PNODE, s0[e].node, m.node, 0, {}};
                for (size_t i = 0; i < ks.size(); ++i) r.f[s0[e].kids[i]] = at.at(ks[i]);
                rels.push_back(r);
            }
        }
    }
    return true;
}

}  // namespace

namespace edb {

void pq_layout(const edb_graph& g, const struct edb_schedule& s, const edb_operand_shape* shapes,
               std::vector<int32_t>& slot_of, std::map<std::tuple<int, int, int>, int32_t>& pad_of,
               std::vector<int32_t>& lead) {
    const int V = g.V;
    const int B = (int)s.batch_type.size();
    const int32_t* bptr = s.batch_ptr.data();
    int n = V;
    pad_of.clear();
    std::vector<std::vector<std::vector<int>>> operands(B);
    std::vector<std::vector<int>> ids(B);   // 0 the rows, 1 + p positional child p
    std::vector<std::vector<int>> ragged(B);
    for (int b = 0; b < B; ++b) {
        const edb_operand_shape& sh = shapes[s.batch_type[b]];
        std::vector<int> rows(s.batch_nodes.begin() + bptr[b], s.batch_nodes.begin() + bptr[b + 1]);
        operands[b].push_back(rows);
        ids[b].push_back(0);
        for (int p = 0; p < sh.n_fixed; ++p) {
            bool any = false;
            for (int v : rows) any |= g.child_idx[g.child_ptr[v] + p] >= 0;
            if (!any) continue;
            std::vector<int> vars;
            for (int v : rows) {
                int c = g.child_idx[g.child_ptr[v] + p];
                if (c < 0) {
                    pad_of[{b, p, v}] = n;
                    c = n++;
                }
                vars.push_back(c);
            }
            std::set<int> uniq(vars.begin(), vars.end());
            if (uniq.size() == vars.size()) {
                operands[b].push_back(vars);
                ids[b].push_back(1 + p);
            }
        }
        if (sh.ragged) {
            std::vector<int> rl;
            for (int v : rows)
                for (int64_t e = g.child_ptr[v] + sh.n_fixed; e < g.child_ptr[v + 1]; ++e)
                    if (g.child_idx[e] >= 0) rl.push_back(g.child_idx[e]);
            std::set<int> uniq(rl.begin(), rl.end());
            if (rl.size() >= 2 && uniq.size() == rl.size()) ragged[b] = rl;
        }
    }
    PQTree t(n);
    // group[b]: (operand index) of the operands taking part in alignment
    std::vector<std::vector<int>> group(B);
    bool ch;
    for (int b = B - 1; b >= 0; --b) {
        for (size_t i = 1; i < operands[b].size(); ++i)
            if (t.reduce(operands[b][i], &ch)) group[b].push_back((int)i);
        if (!ragged[b].empty()) t.reduce(ragged[b], &ch);
        if (t.reduce(operands[b][0], &ch)) group[b].insert(group[b].begin(), 0);
    }
    lead.assign(B, 0);
    for (int b = 0; b < B; ++b) lead[b] = group[b].empty() ? 0 : ids[b][group[b][0]];
    auto active = [&](int b) {
        return group[b].size() >= 2 && operands[b][group[b][0]].size() >= 2;
    };
    auto ops_of = [&](int b) {
        std::vector<const std::vector<int>*> o;
        for (int i : group[b]) o.push_back(&operands[b][i]);
        return o;
    };
    std::vector<std::vector<int>> cons;
    for (;;) {
        bool changed = false;
        for (int b = 0; b < B; ++b) {
            if (!active(b)) continue;
            parse_constraints(t, ops_of(b), cons);
            for (const std::vector<int>& c : cons) {
                if (!t.reduce(c, &ch)) {
                    group[b].resize(1);
                    break;
                }
                changed |= ch;
            }
        }
        if (!changed) break;
    }
    UnionFind uf(t);
    std::vector<Relation> rels;
    for (int b = 0; b < B; ++b) {
        if (!active(b)) continue;
        if (!relations(t, ops_of(b), rels)) continue;
        for (const Relation& r : rels) {
            if (r.kind == QNODE) uf.union_q(r.x, r.y, r.parity);
            else uf.union_p(r.x, r.y, r.f);
        }
    }
    // leaf order
    slot_of.assign(n, 0);
    int32_t next = 1;
    std::vector<int> stack;
    if (t.root >= 0) stack.push_back(t.root);
    std::map<int, int> T;
    while (!stack.empty()) {
        const int x = stack.back();
        stack.pop_back();
        if (t.kind[x] == LEAF) {
            slot_of[x] = next++;
            continue;
        }
        std::vector<int> kids;
        if (t.order_kind(x) == QNODE) {
            int parity;
            uf.find_q(x, &parity);
            kids = t.children[x];
            if (parity) std::reverse(kids.begin(), kids.end());
        } else {
            const int r = uf.find_p(x, T);
            for (int c : t.children[r]) kids.push_back(T.at(c));
        }
        for (auto it = kids.rbegin(); it != kids.rend(); ++it) stack.push_back(*it);
    }
}

}  // namespace edb
