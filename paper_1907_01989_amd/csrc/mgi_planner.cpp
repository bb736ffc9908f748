// Intermediate-tensor planner (Sec. 5 of the paper).
//
// Greedy shared objects (Algorithm 1): operators are visited in execution
// order.  Each intermediate output of an operator takes a new shared object if
// the pool of free objects is empty, otherwise the free object closest in size
// to the tensor (absolute difference), which grows to the tensor's size when
// smaller.  After all outputs of the operator are placed, every intermediate
// input whose last consumer is this operator returns its object to the pool.
// Placing outputs before freeing inputs keeps an operator's output from
// sharing memory with its own input.
//
// The pool is an ordered multimap keyed by object size (the binary search tree
// of the paper) so "closest size" is a lower_bound plus one step back:
// O(n log n) over n tensors.  Equal distances go to the lower object index;
// the set of live objects needs no explicit container because an object is
// either in the pool or attached to a live tensor.
//
// Minimum-cost flow (Sec. 5, flow-network paragraph): a source s, a sink t,
// and vertices l_x, r_x per tensor x; unit-capacity edges s -> r_x of cost
// size_x (a new object for x), l_x -> r_y of cost max(0, size_y - size_x)
// whenever x's last use precedes y's producer (y takes over x's object),
// s -> l_x and r_x -> t of cost 0.  A flow of value n of minimum cost is built
// by n successive shortest augmenting paths, each found with SPFA (a
// queue-driven Bellman-Ford, needed because residual edges carry negative
// costs).  Saturated s -> r_x edges open objects, saturated l_x -> r_y edges
// chain y behind x; an object's size is the largest tensor in its chain.
#include <algorithm>
#include <cstdint>
#include <deque>
#include <limits>
#include <map>
#include <numeric>

#include "mgi_internal.h"

namespace mgi {

PlanResult plan_naive(const std::vector<size_t> &sizes) {
    PlanResult r;
    r.object_of.resize(sizes.size());
    for (size_t t = 0; t < sizes.size(); ++t) {
        r.object_of[t] = (int)t;
        r.object_size.push_back(sizes[t]);
    }
    return r;
}

PlanResult plan_greedy(const std::vector<size_t> &sizes, const std::vector<int> &first,
                       const std::vector<int> &last) {
    const int n = (int)sizes.size();
    PlanResult r;
    r.object_of.assign(n, -1);
    int max_op = -1;
    for (int t = 0; t < n; ++t) max_op = std::max(max_op, std::max(first[t], last[t]));
    // tensors produced / released at each operator, in tensor order
    std::vector<std::vector<int>> produced(max_op + 1), released(max_op + 1);
    for (int t = 0; t < n; ++t) {
        produced[first[t]].push_back(t);
        if (last[t] >= 0) released[last[t]].push_back(t);
    }
    // pool of free objects: size -> object index (ordered by size, then index)
    std::multimap<size_t, int> pool;
    auto pool_erase = [&](std::multimap<size_t, int>::iterator it) { pool.erase(it); };
    for (int op = 0; op <= max_op; ++op) {
        for (int t : produced[op]) {
            const size_t sz = sizes[t];
            int k;
            if (pool.empty()) {
                k = (int)r.object_size.size();
                r.object_size.push_back(sz);
            } else {
                // candidates: the smallest object >= sz and the largest object < sz;
                // among equal sizes the multimap keeps insertion order, so scan the
                // run of equal keys for the lowest index.
                auto hi = pool.lower_bound(sz);
                std::multimap<size_t, int>::iterator best = pool.end();
                auto better = [&](std::multimap<size_t, int>::iterator c) {
                    if (best == pool.end()) return true;
                    size_t dc = c->first > sz ? c->first - sz : sz - c->first;
                    size_t db = best->first > sz ? best->first - sz : sz - best->first;
                    return dc < db || (dc == db && c->second < best->second);
                };
                if (hi != pool.end()) {
                    for (auto it = hi; it != pool.end() && it->first == hi->first; ++it)
                        if (better(it)) best = it;
                }
                if (hi != pool.begin()) {
                    auto lo = std::prev(hi);
                    const size_t key = lo->first;
                    for (auto it = pool.lower_bound(key); it != pool.end() && it->first == key; ++it)
                        if (better(it)) best = it;
                }
                k = best->second;
                pool_erase(best);
                if (sz > r.object_size[k]) r.object_size[k] = sz;
            }
            r.object_of[t] = k;
        }
        for (int t : released[op]) {
            const int k = r.object_of[t];
            pool.emplace(r.object_size[k], k);
        }
    }
    return r;
}

PlanResult plan_mcfp(const std::vector<size_t> &sizes, const std::vector<int> &first,
                     const std::vector<int> &last) {
    const int n = (int)sizes.size();
    // tensors in order of production (ties by index); a tensor nothing
    // consumes is dead right after its producer
    std::vector<int> ts(n);
    std::iota(ts.begin(), ts.end(), 0);
    std::stable_sort(ts.begin(), ts.end(), [&](int a, int b) { return first[a] < first[b]; });
    auto end_of = [&](int t) { return last[t] < 0 ? first[t] : last[t]; };

    struct Edge {
        int to, cap;
        int64_t cost;
    };
    const int S = 0, T = 1, nv = 2 + 2 * n;
    auto L = [](int i) { return 2 + 2 * i; };
    auto R = [](int i) { return 3 + 2 * i; };
    std::vector<Edge> edges;
    std::vector<std::vector<int>> adj(nv);
    auto add = [&](int u, int v, int64_t cost) {
        adj[u].push_back((int)edges.size());
        edges.push_back({v, 1, cost});
        adj[v].push_back((int)edges.size());
        edges.push_back({u, 0, -cost});
        return (int)edges.size() - 2;
    };
    std::vector<int> new_edge(n);
    for (int i = 0; i < n; ++i) new_edge[i] = add(S, R(i), (int64_t)sizes[ts[i]]);
    std::vector<std::vector<std::pair<int, int>>> into(n);   // (source position, edge) per target
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < n; ++j)
            if (end_of(ts[i]) < first[ts[j]]) {
                const int64_t c = sizes[ts[j]] > sizes[ts[i]] ? (int64_t)(sizes[ts[j]] - sizes[ts[i]]) : 0;
                into[j].push_back({i, add(L(i), R(j), c)});
            }
    for (int i = 0; i < n; ++i) add(S, L(i), 0);
    for (int i = 0; i < n; ++i) add(R(i), T, 0);

    const int64_t INF = std::numeric_limits<int64_t>::max() / 4;
    std::vector<int64_t> dist(nv);
    std::vector<int> pred(nv);
    std::vector<char> queued(nv);
    for (int k = 0; k < n; ++k) {
        std::fill(dist.begin(), dist.end(), INF);
        std::fill(pred.begin(), pred.end(), -1);
        std::fill(queued.begin(), queued.end(), 0);
        std::deque<int> q;
        dist[S] = 0;
        q.push_back(S);
        queued[S] = 1;
        while (!q.empty()) {
            const int u = q.front();
            q.pop_front();
            queued[u] = 0;
            for (int e : adj[u]) {
                const Edge &ed = edges[e];
                if (ed.cap > 0 && dist[u] + ed.cost < dist[ed.to]) {
                    dist[ed.to] = dist[u] + ed.cost;
                    pred[ed.to] = e;
                    if (!queued[ed.to]) {
                        queued[ed.to] = 1;
                        q.push_back(ed.to);
                    }
                }
            }
        }
        // every r_x still reaches t, and s -> r_x is open while r_x -> t is
        for (int v = T; v != S;) {
            const int e = pred[v];
            edges[e].cap -= 1;
            edges[e ^ 1].cap += 1;
            v = edges[e ^ 1].to;
        }
    }

    PlanResult r;
    r.object_of.assign(n, -1);
    for (int j = 0; j < n; ++j) {
        const int y = ts[j];
        int k = -1;
        if (edges[new_edge[j]].cap == 0) {
            k = (int)r.object_size.size();
            r.object_size.push_back(sizes[y]);
        } else {
            for (const auto &pe : into[j])
                if (edges[pe.second].cap == 0) k = r.object_of[ts[pe.first]];
            r.object_size[k] = std::max(r.object_size[k], sizes[y]);
        }
        r.object_of[y] = k;
    }
    return r;
}

}  // namespace mgi

using namespace mgi;

extern "C" mgi_status mgi_planner_assign(int planner, int n_tensors, const size_t *sizes,
                                         const int *first_op, const int *last_op, int *object_of,
                                         size_t *object_sizes, int *n_objects) {
    MGI_ABI_TRY
    if (n_tensors < 0) return fail(MGI_ERR_INVALID_ARG, "mgi_planner_assign: n_tensors < 0");
    if (n_tensors > 0 && (!sizes || !first_op || !last_op || !object_of || !object_sizes))
        return fail(MGI_ERR_INVALID_ARG, "mgi_planner_assign: null pointer");
    if (!n_objects) return fail(MGI_ERR_INVALID_ARG, "mgi_planner_assign: null n_objects");
    std::vector<size_t> sz(sizes, sizes + n_tensors);
    std::vector<int> fi(first_op, first_op + n_tensors), la(last_op, last_op + n_tensors);
    for (int t = 0; t < n_tensors; ++t) {
        if (fi[t] < 0 || (la[t] >= 0 && la[t] < fi[t]))
            return fail(MGI_ERR_INVALID_ARG, "mgi_planner_assign: tensor " + std::to_string(t) +
                                                 " has an invalid lifetime");
    }
    PlanResult r;
    if (planner == MGI_PLANNER_NAIVE) r = plan_naive(sz);
    else if (planner == MGI_PLANNER_GREEDY) r = plan_greedy(sz, fi, la);
    else if (planner == MGI_PLANNER_MCFP) r = plan_mcfp(sz, fi, la);
    else return fail(MGI_ERR_UNSUPPORTED, "mgi_planner_assign: unknown planner");
    for (int t = 0; t < n_tensors; ++t) object_of[t] = r.object_of[t];
    for (size_t k = 0; k < r.object_size.size(); ++k) object_sizes[k] = r.object_size[k];
    *n_objects = (int)r.object_size.size();
    return MGI_OK;
    MGI_ABI_CATCH("mgi_planner_assign")
}
