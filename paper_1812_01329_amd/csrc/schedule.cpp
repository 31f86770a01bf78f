// Host-side integer schedules and validation.
//
// Sequences: the running rows of a loop whose trip count differs per
// sequence (Figure 1 loop, Section 4.2.1).  Sorting the batch by length,
// longest first, makes the rows still running at step t a prefix of the
// sorted order, so step t works on a dense block of active[t] rows.
//
// Trees: the recursion of the TreeNN programs (Section 6.1, footnote 6)
// turned into frontiers: a node's level is its height above the leaves, and
// all nodes of one level are independent cell applications that run as one
// batched contraction (the parallel execution of independent operations,
// Section 6.3.1 "+PARL").
//
// All checks run before any device work so that a rejected call writes
// nothing (all-or-nothing updates, Section 3.2).
#include "runtime.hpp"

#include <algorithm>
#include <cstring>
#include <vector>

namespace janus {

janus_status build_seq_schedule(int32_t B, int32_t T, const int32_t* lengths, SeqSchedule& s) {
    if (B <= 0 || T < 0) return JANUS_ERR_INVALID_ARG;
    s.B = B;
    s.T = T;
    std::vector<int32_t> len(B, T);
    if (lengths) {
        for (int32_t b = 0; b < B; ++b) {
            if (lengths[b] < 0 || lengths[b] > T) return JANUS_ERR_LENGTH;
            len[b] = lengths[b];
        }
    }
    // counting sort by length, longest first, ties by batch index
    std::vector<int32_t> count(T + 2, 0);
    for (int32_t b = 0; b < B; ++b) count[len[b]]++;
    std::vector<int32_t> start(T + 2, 0);   // start[v] = #{b : len_b > v}
    int32_t acc = 0;
    for (int32_t v = T; v >= 0; --v) {
        start[v] = acc;
        acc += count[v];
    }
    s.perm.assign(B, 0);
    {
        std::vector<int32_t> fill(start.begin(), start.end());
        for (int32_t b = 0; b < B; ++b) s.perm[fill[len[b]]++] = b;
    }
    s.t_eff = 0;
    for (int32_t b = 0; b < B; ++b) s.t_eff = std::max(s.t_eff, len[b]);
    s.active.assign(T + 1, 0);               // active[T] = 0 sentinel
    for (int32_t t = 0; t < s.t_eff; ++t) s.active[t] = start[t];
    s.offsets.assign(T + 2, 0);
    for (int32_t t = 0; t <= T; ++t) s.offsets[t + 1] = s.offsets[t] + s.active[t];
    s.fixed = true;
    for (int32_t b = 0; b < B; ++b) s.fixed = s.fixed && (len[b] == T);
    s.packed = s.offsets[T];
    if (!s.fixed) {
        // row of x (index into [T*B]) and row of the previous h for every packed row
        s.xrow.assign(std::max<int64_t>(s.packed, 1), 0);
        s.prevrow.assign(std::max<int64_t>(s.packed, 1), 0);
        for (int32_t t = 0; t < s.t_eff; ++t) {
            for (int32_t r = 0; r < s.active[t]; ++r) {
                int64_t p = s.offsets[t] + r;
                s.xrow[p] = t * B + s.perm[r];
                s.prevrow[p] = (t == 0) ? r : B + s.offsets[t - 1] + r;
            }
        }
    }
    return JANUS_OK;
}

janus_status validate_tree_batch(const janus_tree_batch* t, int32_t V) {
    if (!t || !t->left || !t->right || !t->word || !t->root) return JANUS_ERR_INVALID_ARG;
    const int32_t N = t->num_nodes;
    if (N <= 0 || t->num_trees <= 0) return JANUS_ERR_INVALID_ARG;
    std::vector<int32_t> parents(N, 0);
    for (int32_t n = 0; n < N; ++n) {
        const int32_t l = t->left[n], r = t->right[n];
        if ((l < 0) != (r < 0)) return JANUS_ERR_TREE;
        if (l < 0) {
            if (l != -1 || r != -1) return JANUS_ERR_TREE;
            if (t->word[n] < 0 || t->word[n] >= V) return JANUS_ERR_TOKEN;
        } else {
            if (l >= N || r >= N || l == r) return JANUS_ERR_TREE;
            if (t->word[n] != -1) return JANUS_ERR_TREE;
            parents[l]++;
            parents[r]++;
        }
    }
    for (int32_t n = 0; n < N; ++n)
        if (parents[n] > 1) return JANUS_ERR_TREE;
    std::vector<char> is_root(N, 0);
    for (int32_t k = 0; k < t->num_trees; ++k) {
        const int32_t r = t->root[k];
        if (r < 0 || r >= N || parents[r] != 0 || is_root[r]) return JANUS_ERR_TREE;
        is_root[r] = 1;
    }
    // reachability: with one parent per node and parentless roots, a node
    // outside every root's subtree lies on a cycle or a stray component
    std::vector<int32_t> stack;
    stack.reserve(N);
    int64_t reached = 0;
    for (int32_t k = 0; k < t->num_trees; ++k) stack.push_back(t->root[k]);
    while (!stack.empty()) {
        const int32_t n = stack.back();
        stack.pop_back();
        if (++reached > N) return JANUS_ERR_TREE;
        if (t->left[n] >= 0) {
            stack.push_back(t->left[n]);
            stack.push_back(t->right[n]);
        }
    }
    if (reached != N) return JANUS_ERR_TREE;
    return JANUS_OK;
}

janus_status build_tree_schedule(const janus_tree_batch* t, int32_t V, TreeSchedule& s) {
    janus_status st = validate_tree_batch(t, V);
    if (st != JANUS_OK) return st;
    const int32_t N = t->num_nodes;
    s.N = N;
    s.num_trees = t->num_trees;
    s.level.assign(N, -1);
    // heights by an explicit post-order walk from every root
    std::vector<std::pair<int32_t, int32_t>> stack;   // (node, state)
    for (int32_t k = 0; k < t->num_trees; ++k) {
        stack.push_back({t->root[k], 0});
        while (!stack.empty()) {
            auto& top = stack.back();
            const int32_t n = top.first;
            if (t->left[n] < 0) {
                s.level[n] = 0;
                stack.pop_back();
            } else if (top.second == 0) {
                top.second = 1;
                stack.push_back({t->left[n], 0});
                stack.push_back({t->right[n], 0});
            } else {
                s.level[n] = 1 + std::max(s.level[t->left[n]], s.level[t->right[n]]);
                stack.pop_back();
            }
        }
    }
    int32_t L = 0;
    for (int32_t n = 0; n < N; ++n) L = std::max(L, s.level[n] + 1);
    s.num_levels = L;
    s.level_offsets.assign(L + 1, 0);
    for (int32_t n = 0; n < N; ++n) s.level_offsets[s.level[n] + 1]++;
    for (int32_t k = 0; k < L; ++k) s.level_offsets[k + 1] += s.level_offsets[k];
    s.level_nodes.assign(N, 0);
    s.pos.assign(N, 0);
    {
        std::vector<int32_t> fill(s.level_offsets.begin(), s.level_offsets.end() - 1);
        for (int32_t n = 0; n < N; ++n) {
            const int32_t p = fill[s.level[n]]++;
            s.level_nodes[p] = n;
            s.pos[n] = p;
        }
    }
    s.max_level_size = 0;
    for (int32_t k = 0; k < L; ++k)
        s.max_level_size = std::max(s.max_level_size, s.level_offsets[k + 1] - s.level_offsets[k]);
    return JANUS_OK;
}

janus_status build_nary_schedule(const janus_nary_tree_batch* t, int32_t V, NarySchedule& s) {
    if (!t || t->num_trees <= 0 || t->num_nodes <= 0 || !t->child_offsets || !t->word || !t->root)
        return JANUS_ERR_INVALID_ARG;
    const int32_t N = t->num_nodes, K = t->num_trees;
    const int32_t* off = t->child_offsets;
    if (off[0] != 0) return JANUS_ERR_TREE;
    for (int32_t n = 0; n < N; ++n)
        if (off[n + 1] < off[n]) return JANUS_ERR_TREE;
    const int32_t E = off[N];
    if (E > 0 && !t->children) return JANUS_ERR_INVALID_ARG;
    std::vector<int32_t> parent(N, -1);
    for (int32_t e = 0; e < E; ++e) {
        const int32_t c = t->children[e];
        if (c < 0 || c >= N || parent[c] >= 0) return JANUS_ERR_TREE;
        parent[c] = 1;
    }
    for (int32_t n = 0; n < N; ++n)
        if (t->word[n] < 0 || t->word[n] >= V) return JANUS_ERR_TOKEN;
    // levels by an explicit post-order walk from every root; a node seen twice
    // or never is malformed (a cycle, a shared child, an unreachable node)
    std::vector<int32_t> level(N, -1), state(N, 0), rootk(N, -1);
    std::vector<std::pair<int32_t, int32_t>> stack;
    int32_t seen = 0;
    for (int32_t k = 0; k < K; ++k) {
        const int32_t r = t->root[k];
        if (r < 0 || r >= N || parent[r] >= 0 || state[r] != 0) return JANUS_ERR_TREE;
        rootk[r] = k;
        stack.push_back({r, off[r]});
        state[r] = 1;
        while (!stack.empty()) {
            auto& [n, next] = stack.back();
            if (next < off[n + 1]) {
                const int32_t c = t->children[next++];
                if (state[c] != 0) return JANUS_ERR_TREE;
                state[c] = 1;
                stack.push_back({c, off[c]});
            } else {
                int32_t lv = 0;
                for (int32_t e = off[n]; e < off[n + 1]; ++e) lv = std::max(lv, level[t->children[e]] + 1);
                level[n] = lv;
                state[n] = 2;
                ++seen;
                stack.pop_back();
            }
        }
    }
    if (seen != N) return JANUS_ERR_TREE;
    int32_t L = 0;
    for (int32_t n = 0; n < N; ++n) L = std::max(L, level[n] + 1);
    s.N = N;
    s.level_offsets.assign(L + 1, 0);
    for (int32_t n = 0; n < N; ++n) ++s.level_offsets[level[n] + 1];
    for (int32_t k = 0; k < L; ++k) s.level_offsets[k + 1] += s.level_offsets[k];
    std::vector<int32_t> pos(N), fill(s.level_offsets.begin(), s.level_offsets.end() - 1);
    for (int32_t n = 0; n < N; ++n) pos[n] = fill[level[n]]++;   // ascending id within a level
    s.pword.assign(N, 0);
    s.rootk.assign(N, -1);
    s.rootpos.assign(K, 0);
    s.pcoff.assign(N + 1, 0);
    std::vector<int32_t> node_at(N);
    for (int32_t n = 0; n < N; ++n) node_at[pos[n]] = n;
    for (int32_t p = 0; p < N; ++p) {
        const int32_t n = node_at[p];
        s.pword[p] = t->word[n];
        s.rootk[p] = rootk[n];
        s.pcoff[p + 1] = s.pcoff[p] + (off[n + 1] - off[n]);
    }
    s.pkids.assign(std::max(E, 1), 0);
    for (int32_t p = 0; p < N; ++p) {
        const int32_t n = node_at[p];
        for (int32_t e = off[n], q = s.pcoff[p]; e < off[n + 1]; ++e, ++q) s.pkids[q] = pos[t->children[e]];
    }
    for (int32_t k = 0; k < K; ++k) s.rootpos[k] = pos[t->root[k]];
    return JANUS_OK;
}

}  // namespace janus

extern "C" janus_status janus_lstm_schedule(int32_t B, int32_t T, const int32_t* lengths,
                                            int32_t* perm, int32_t* active, int32_t* offsets,
                                            int32_t* t_eff) {
    if (!lengths || !perm || !active || !offsets || !t_eff) return JANUS_ERR_INVALID_ARG;
    janus::SeqSchedule s;
    janus_status st = janus::build_seq_schedule(B, T, lengths, s);
    if (st != JANUS_OK) return st;
    std::memcpy(perm, s.perm.data(), sizeof(int32_t) * B);
    std::memcpy(active, s.active.data(), sizeof(int32_t) * T);
    std::memcpy(offsets, s.offsets.data(), sizeof(int32_t) * (T + 1));
    *t_eff = s.t_eff;
    return JANUS_OK;
}

extern "C" janus_status janus_tree_schedule_build(const janus_tree_batch* t, int32_t V,
                                                  int32_t* node_level, int32_t* level_offsets,
                                                  int32_t* level_nodes, int32_t* num_levels) {
    if (!node_level || !level_offsets || !level_nodes || !num_levels) return JANUS_ERR_INVALID_ARG;
    janus::TreeSchedule s;
    janus_status st = janus::build_tree_schedule(t, V, s);
    if (st != JANUS_OK) return st;
    std::memcpy(node_level, s.level.data(), sizeof(int32_t) * s.N);
    std::memcpy(level_offsets, s.level_offsets.data(), sizeof(int32_t) * (s.num_levels + 1));
    std::memcpy(level_nodes, s.level_nodes.data(), sizeof(int32_t) * s.N);
    *num_levels = s.num_levels;
    return JANUS_OK;
}
