// graph.hip -- topology-aware subgraph matching of two computational graphs
// (Section 4.2), host code.
//
// Dominators by the iterative algorithm of Cooper, Harvey and Kennedy ("A
// Simple, Fast Dominance Algorithm", 2001) over the reverse postorder of the
// region, dominance queries by entry/exit times of the dominator tree, the
// cut chain by a longest-chain table built backwards and a greedy walk that
// takes the smallest admissible next point (the lexicographically smallest of
// the longest chains), and the regions between consecutive cuts matched
// recursively.

#include <algorithm>
#include <cstdint>
#include <vector>

#include "mag_internal.hpp"

namespace mag {

namespace {

struct Graph {
    int n = 0;
    std::vector<int> off, adj;    // successors (CSR)
    std::vector<int> poff, padj;  // predecessors
};

void build(const mag_graph& g, Graph& out)
{
    const int n = g.n_nodes;
    out.n = n;
    out.off.assign(n + 1, 0);
    out.poff.assign(n + 1, 0);
    for (int e = 0; e < g.n_edges; ++e) {
        ++out.off[g.src[e] + 1];
        ++out.poff[g.dst[e] + 1];
    }
    for (int v = 0; v < n; ++v) {
        out.off[v + 1] += out.off[v];
        out.poff[v + 1] += out.poff[v];
    }
    out.adj.assign(g.n_edges, 0);
    out.padj.assign(g.n_edges, 0);
    std::vector<int> a(out.off.begin(), out.off.end() - 1), b(out.poff.begin(), out.poff.end() - 1);
    for (int e = 0; e < g.n_edges; ++e) {
        out.adj[a[g.src[e]]++] = g.dst[e];
        out.padj[b[g.dst[e]]++] = g.src[e];
    }
}

// dominator tree of a region (its nodes listed in `nodes`, loc[v] = the local
// index of node v or -1 outside) from its entry s; arrays are local
struct Dom {
    std::vector<int> idom, tin, tout;  // by local index; tin < 0: unreachable
    bool dominates(int d, int v) const { return tin[d] <= tin[v] && tout[v] <= tout[d]; }
};

void dominators(const Graph& g, const std::vector<int>& nodes, const std::vector<int>& loc, int s,
                Dom& D)
{
    const int n = (int)nodes.size();
    std::vector<int> order, rpo(n, -1), it(n, 0), stack;
    std::vector<char> seen(n, 0);
    const int ls = loc[s];
    stack.push_back(ls);  // postorder by an explicit stack (local indices)
    seen[ls] = 1;
    while (!stack.empty()) {
        const int u = stack.back();
        const int gu = nodes[u];
        bool pushed = false;
        while (it[u] < g.off[gu + 1] - g.off[gu]) {
            const int v = loc[g.adj[g.off[gu] + it[u]++]];
            if (v >= 0 && !seen[v]) {
                seen[v] = 1;
                stack.push_back(v);
                pushed = true;
                break;
            }
        }
        if (!pushed) {
            order.push_back(u);
            stack.pop_back();
        }
    }
    std::reverse(order.begin(), order.end());
    for (int i = 0; i < (int)order.size(); ++i) rpo[order[i]] = i;
    std::vector<int>& idom = D.idom;
    idom.assign(n, -1);
    idom[ls] = ls;
    for (bool changed = true; changed;) {
        changed = false;
        for (int i = 1; i < (int)order.size(); ++i) {
            const int b = order[i];
            const int gb = nodes[b];
            int nd = -1;
            for (int q = g.poff[gb]; q < g.poff[gb + 1]; ++q) {
                const int p = loc[g.padj[q]];
                if (p < 0 || rpo[p] < 0 || idom[p] < 0) continue;
                if (nd < 0) {
                    nd = p;
                    continue;
                }
                int x = p, y = nd;  // the nearest common dominator
                while (x != y) {
                    while (rpo[x] > rpo[y]) x = idom[x];
                    while (rpo[y] > rpo[x]) y = idom[y];
                }
                nd = x;
            }
            if (nd >= 0 && idom[b] != nd) {
                idom[b] = nd;
                changed = true;
            }
        }
    }
    // entry / exit times of the dominator tree
    std::vector<int> coff(n + 1, 0), kids;
    for (int v : order)
        if (v != ls) ++coff[idom[v] + 1];
    for (int v = 0; v < n; ++v) coff[v + 1] += coff[v];
    kids.assign(coff[n], 0);
    std::vector<int> fill(coff.begin(), coff.end() - 1);
    for (int v : order)
        if (v != ls) kids[fill[idom[v]]++] = v;
    D.tin.assign(n, -1);
    D.tout.assign(n, -2);
    int clock = 0;
    std::vector<int> pos(n, 0);
    stack.assign(1, ls);
    D.tin[ls] = clock++;
    while (!stack.empty()) {
        const int u = stack.back();
        if (pos[u] < coff[u + 1] - coff[u]) {
            const int v = kids[coff[u] + pos[u]++];
            D.tin[v] = clock++;
            stack.push_back(v);
        } else {
            D.tout[u] = clock++;
            stack.pop_back();
        }
    }
}

// the dominator path s .. t (t's dominators, s first), local indices
std::vector<int> dom_path(const Dom& D, int ls, int lt)
{
    std::vector<int> p;
    for (int v = lt;; v = D.idom[v]) {
        p.push_back(v);
        if (v == ls) break;
    }
    std::reverse(p.begin(), p.end());
    return p;
}

struct Matcher {
    const Graph& g1;
    const Graph& g2;
    std::vector<int32_t>& out;
    std::vector<int> loc1, loc2;  // global -> local index of the current region, else -1

    void rec(const std::vector<int>& nodes1, int s1, int e1, const std::vector<int>& nodes2, int s2,
             int e2, const std::vector<std::pair<int, int>>& eq)
    {
        for (int i = 0; i < (int)nodes1.size(); ++i) loc1[nodes1[i]] = i;
        for (int i = 0; i < (int)nodes2.size(); ++i) loc2[nodes2[i]] = i;
        Dom D1, D2;
        dominators(g1, nodes1, loc1, s1, D1);
        dominators(g2, nodes2, loc2, s2, D2);
        const std::vector<int> p1 = dom_path(D1, loc1[s1], loc1[e1]);
        const std::vector<int> p2 = dom_path(D2, loc2[s2], loc2[e2]);
        std::vector<int> pos1(nodes1.size(), -1), pos2(nodes2.size(), -1);
        for (int i = 0; i < (int)p1.size(); ++i) pos1[p1[i]] = i;
        for (int j = 0; j < (int)p2.size(); ++j) pos2[p2[j]] = j;
        std::vector<std::pair<int, int>> pts;
        for (const auto& q : eq) {
            const int a = loc1[q.first], b = loc2[q.second];
            if (a >= 0 && b >= 0 && pos1[a] >= 0 && pos2[b] >= 0) pts.push_back({pos1[a], pos2[b]});
        }
        const std::pair<int, int> first{0, 0}, last{(int)p1.size() - 1, (int)p2.size() - 1};
        pts.push_back(first);
        pts.push_back(last);
        std::sort(pts.begin(), pts.end());
        pts.erase(std::unique(pts.begin(), pts.end()), pts.end());
        // longest chain from each point to the last one (-1: none)
        const int P = (int)pts.size();
        std::vector<int> len(P, -1);
        for (int k = P - 1; k >= 0; --k) {
            if (pts[k] == last) {
                len[k] = 1;
                continue;
            }
            for (int q = k + 1; q < P; ++q)
                if (pts[q].first > pts[k].first && pts[q].second > pts[k].second && len[q] > 0)
                    len[k] = std::max(len[k], len[q] + 1);
        }
        std::vector<std::pair<int, int>> cuts;  // global node ids
        int k = 0;  // (0, 0) is the smallest point
        cuts.push_back({nodes1[p1[pts[k].first]], nodes2[p2[pts[k].second]]});
        while (pts[k] != last) {
            int nxt = -1;
            for (int q = k + 1; q < P && nxt < 0; ++q)  // the smallest admissible next point
                if (pts[q].first > pts[k].first && pts[q].second > pts[k].second &&
                    len[q] == len[k] - 1)
                    nxt = q;
            k = nxt;
            cuts.push_back({nodes1[p1[pts[k].first]], nodes2[p2[pts[k].second]]});
        }
        if (cuts.size() <= 2) {
            for (int v : nodes1) loc1[v] = -1;
            for (int v : nodes2) loc2[v] = -1;
            out.insert(out.end(), {s1, e1, s2, e2});
            return;
        }
        // the regions between consecutive cuts, and the eq pairs inside each
        const size_t R = cuts.size() - 1;
        std::vector<std::vector<int>> r1(R), r2(R);
        auto region_of = [&](const Dom& D, const std::vector<int>& loc,
                             const std::vector<std::pair<int, int>>& cs, bool second, int v) {
            // the last cut dominating v; v belongs to the region starting there,
            // and a cut node also ends the region before it
            int lo = 0, hi = (int)R;  // cuts[lo] dominates v (the entry dominates everything)
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                const int c = second ? cs[mid].second : cs[mid].first;
                if (D.dominates(loc[c], loc[v])) lo = mid; else hi = mid - 1;
            }
            return lo;
        };
        for (int v : nodes1) {
            const int lv = loc1[v];
            if (D1.tin[lv] < 0) continue;
            const int r = region_of(D1, loc1, cuts, false, v);
            if (r < (int)R) r1[r].push_back(v);
            if (r > 0 && cuts[r].first == v) r1[r - 1].push_back(v);
        }
        for (int v : nodes2) {
            const int lv = loc2[v];
            if (D2.tin[lv] < 0) continue;
            const int r = region_of(D2, loc2, cuts, true, v);
            if (r < (int)R) r2[r].push_back(v);
            if (r > 0 && cuts[r].second == v) r2[r - 1].push_back(v);
        }
        std::vector<std::vector<std::pair<int, int>>> sub(R);
        {
            // region index of each node (entries; exits are checked by id)
            for (size_t r = 0; r < R; ++r)
                for (int v : r1[r]) loc1[v] = (int)r;
            for (size_t r = 0; r < R; ++r)
                for (int v : r2[r]) loc2[v] = (int)r;
            for (const auto& q : eq) {
                const int a = loc1[q.first], b = loc2[q.second];
                if (a >= 0 && a == b) sub[a].push_back(q);
            }
        }
        for (int v : nodes1) loc1[v] = -1;
        for (int v : nodes2) loc2[v] = -1;
        for (size_t r = 0; r < R; ++r)
            rec(r1[r], cuts[r].first, cuts[r + 1].first, r2[r], cuts[r].second,
                cuts[r + 1].second, sub[r]);
    }
};

// a DAG on which every node lies on a path from node 0 to node n-1
bool well_formed(const Graph& g)
{
    const int n = g.n;
    std::vector<int> indeg(n, 0), q;
    for (int v = 0; v < n; ++v) indeg[v] = g.poff[v + 1] - g.poff[v];
    for (int v = 0; v < n; ++v)
        if (indeg[v] == 0) q.push_back(v);
    size_t h = 0;
    while (h < q.size()) {
        const int u = q[h++];
        for (int e = g.off[u]; e < g.off[u + 1]; ++e)
            if (--indeg[g.adj[e]] == 0) q.push_back(g.adj[e]);
    }
    if ((int)q.size() != n) return false;  // a cycle
    std::vector<char> fwd(n, 0), bwd(n, 0);
    std::vector<int> st{0};
    fwd[0] = 1;
    while (!st.empty()) {
        const int u = st.back();
        st.pop_back();
        for (int e = g.off[u]; e < g.off[u + 1]; ++e)
            if (!fwd[g.adj[e]]) fwd[g.adj[e]] = 1, st.push_back(g.adj[e]);
    }
    st.assign(1, n - 1);
    bwd[n - 1] = 1;
    while (!st.empty()) {
        const int u = st.back();
        st.pop_back();
        for (int e = g.poff[u]; e < g.poff[u + 1]; ++e)
            if (!bwd[g.padj[e]]) bwd[g.padj[e]] = 1, st.push_back(g.padj[e]);
    }
    for (int v = 0; v < n; ++v)
        if (!fwd[v] || !bwd[v]) return false;
    return true;
}

}  // namespace

// 0 on success, else the library status code (the caller sets the message)
int match_subgraphs(const mag_graph& a, const mag_graph& b, const int32_t* eq, int32_t n_eq,
                    std::vector<int32_t>& out)
{
    Graph g1, g2;
    build(a, g1);
    build(b, g2);
    if (!well_formed(g1) || !well_formed(g2)) return MAG_E_GRAPH;
    std::vector<std::pair<int, int>> pairs;
    for (int32_t p = 0; p < n_eq; ++p) pairs.push_back({eq[2 * p], eq[2 * p + 1]});
    std::vector<int> all1(g1.n), all2(g2.n);
    for (int v = 0; v < g1.n; ++v) all1[v] = v;
    for (int v = 0; v < g2.n; ++v) all2[v] = v;
    Matcher m{g1, g2, out, std::vector<int>(g1.n, -1), std::vector<int>(g2.n, -1)};
    m.rec(all1, 0, g1.n - 1, all2, 0, g2.n - 1, pairs);
    return MAG_OK;
}

}  // namespace mag
