// Speculative beam-search controller (host, exact): early pruning (Sec. 4.1) and lazy
// verification (Sec. 4.3).
//
// The search keeps, at every depth (reasoning step), the top k candidates by verifier score, and
// each kept candidate expands into the next step's candidates (beam search, Sec. 2.2).  Under
// speculation a candidate expands as soon as its own score is known, before its round is decided,
// so candidates of several depths are in flight at once.
//
// Membership.  The members of round d are the children of round d-1's selected candidates (the
// roots for d = 0).  While round d-1 is undecided every depth-d candidate is speculative: it is a
// member only if its parent is selected, and then so are its siblings.
//
// Early pruning.  A scored candidate is pruned when at least k candidates that are surely in its
// round (if it is) have strictly higher scores: it can no longer reach the top k (rule 1).  Once k
// candidates surely in the round reach the perfect score 1.0, the first k of them (in score
// arrival order) are the round's selection and every other candidate of the round is pruned (rule
// 2).  For a speculative candidate "surely in its round" means its sibling group; for a member it
// means the whole round.  A round is decided by rule 2, or when every selected parent has expanded
// and every member has a score: the top k by (score descending, arrival ascending) are selected and
// the rest pruned.  Pruning a candidate prunes its subtree.
//
// Lazy verification.  A candidate that completes its step is queued.  The queue should be flushed
// as one verification batch when any of three policies holds: the queued tokens exceed a threshold;
// the sibling group of a queued candidate has completed its step (every unpruned sibling is queued,
// being verified or scored); or a queued candidate has already been deferred max_deferrals times,
// where a deferral is a tick (an iteration of the generator) that passes without a flush.
#include <algorithm>
#include <cstring>
#include <vector>

#include "internal.h"

namespace {

enum : int32_t {
    kGenerating = TKV_CAND_GENERATING,
    kQueued = TKV_CAND_QUEUED,
    kVerifying = TKV_CAND_VERIFYING,
    kVerified = TKV_CAND_VERIFIED,
    kSelected = TKV_CAND_SELECTED,
    kPruned = TKV_CAND_PRUNED
};

struct Node {
    int32_t parent = -1, depth = 0;
    int32_t first_child = -1, n_children = -1;  // n_children -1: not expanded yet
    int32_t state = kGenerating;
    int32_t tokens = 0, deferrals = 0;
    int32_t arrival = -1;  // position of its score in arrival order
    float score = 0.f;
    bool flushed = false, scored = false;
};

}  // namespace

struct tkv_search {
    int32_t k = 1, max_nodes = 0, threshold = 0, max_deferrals = 0;
    int32_t n_roots = -1;  // -1: the roots are not created yet; they are nodes [0, n_roots)
    std::vector<Node> nodes;
    std::vector<int32_t> queue;  // queued candidates in enqueue order
    int64_t queued_tokens = 0;
    int32_t n_arrivals = 0;
    std::vector<uint8_t> decided;               // per depth
    std::vector<std::vector<int32_t>> selected;  // per depth, ascending ids
    std::vector<int32_t> pending;               // pruned since the last tkv_search_pruned
};

using tkv::set_error;

namespace {

bool has_score(const Node& n) { return n.state == kVerified || n.state == kSelected; }

// Ids of the group `parent` heads: the roots for -1, else its children (empty if not expanded).
void group_of(const tkv_search* s, int32_t parent, std::vector<int32_t>& out) {
    out.clear();
    int32_t first = 0, n = s->n_roots;
    if (parent >= 0) {
        first = s->nodes[parent].first_child;
        n = s->nodes[parent].n_children;
    }
    for (int32_t i = 0; i < n; ++i) out.push_back(first + i);
}

void prune_subtree(tkv_search* s, int32_t root) {
    std::vector<int32_t> stack{root};
    while (!stack.empty()) {
        const int32_t x = stack.back();
        stack.pop_back();
        Node& n = s->nodes[x];
        if (n.state == kPruned) continue;
        if (n.state == kQueued) {
            s->queue.erase(std::find(s->queue.begin(), s->queue.end(), x));
            s->queued_tokens -= n.tokens;
        }
        n.state = kPruned;
        s->pending.push_back(x);
        for (int32_t c = 0; c < std::max(0, n.n_children); ++c) stack.push_back(n.first_child + c);
    }
}

// Rule 1 over a set that a candidate of it surely shares: prune every scored candidate that at
// least k others of the set outscore.  Order-independent: the candidates that cause a pruning outrank
// the pruned one and are never pruned by this rule themselves.
bool rank_prune(tkv_search* s, const std::vector<int32_t>& set) {
    std::vector<int32_t> victims;
    for (int32_t x : set) {
        const Node& nx = s->nodes[x];
        if (!has_score(nx)) continue;
        int32_t above = 0;
        for (int32_t y : set)
            if (y != x && has_score(s->nodes[y]) && s->nodes[y].score > nx.score) ++above;
        if (above >= s->k) victims.push_back(x);
    }
    for (int32_t x : victims) prune_subtree(s, x);
    return !victims.empty();
}

// The perfect-scored candidates of a set, in arrival order.
std::vector<int32_t> perfect_by_arrival(const tkv_search* s, const std::vector<int32_t>& set) {
    std::vector<int32_t> p;
    for (int32_t x : set)
        if (has_score(s->nodes[x]) && s->nodes[x].score == 1.0f) p.push_back(x);
    std::sort(p.begin(), p.end(), [s](int32_t a, int32_t b) { return s->nodes[a].arrival < s->nodes[b].arrival; });
    return p;
}

void decide(tkv_search* s, int32_t d, std::vector<int32_t> sel) {
    std::sort(sel.begin(), sel.end());
    s->decided[d] = 1;
    for (int32_t x : sel) s->nodes[x].state = kSelected;
    for (int32_t x = 0; x < static_cast<int32_t>(s->nodes.size()); ++x)
        if (s->nodes[x].depth == d && s->nodes[x].state != kSelected) prune_subtree(s, x);
    s->selected[d] = std::move(sel);
}

// Applies the pruning rules and round decisions until nothing changes.
void settle(tkv_search* s) {
    std::vector<int32_t> members, group;
    for (bool changed = true; changed;) {
        changed = false;
        int32_t max_depth = -1;
        for (const Node& n : s->nodes) max_depth = std::max(max_depth, n.depth);
        if (static_cast<int32_t>(s->decided.size()) <= max_depth) {
            s->decided.resize(max_depth + 1, 0);
            s->selected.resize(max_depth + 1);
        }
        for (int32_t d = 0; d <= max_depth && !changed; ++d) {
            if (s->decided[d]) continue;
            const bool parents_known = d == 0 ? s->n_roots >= 0 : s->decided[d - 1] != 0;
            if (!parents_known) {
                // speculative: each sibling group on its own, under a parent of depth d-1
                for (int32_t p = 0; p < static_cast<int32_t>(s->nodes.size()) && !changed; ++p) {
                    const Node& np = s->nodes[p];
                    if (np.depth != d - 1 || np.state == kPruned || np.n_children <= 0) continue;
                    group.clear();
                    for (int32_t c = 0; c < np.n_children; ++c)
                        if (s->nodes[np.first_child + c].state != kPruned) group.push_back(np.first_child + c);
                    const std::vector<int32_t> perfect = perfect_by_arrival(s, group);
                    if (static_cast<int32_t>(perfect.size()) >= s->k) {  // rule 2 within the group
                        const auto first_k = perfect.begin() + s->k;
                        for (int32_t x : group)
                            if (std::find(perfect.begin(), first_k, x) == first_k) {
                                prune_subtree(s, x);
                                changed = true;
                            }
                    }
                    if (!changed) changed = rank_prune(s, group);  // rule 1 within the group
                }
                continue;
            }
            // members: the roots, or the children of the selected parents
            members.clear();
            bool all_expanded = true;
            if (d == 0) {
                group_of(s, -1, members);
            } else {
                for (int32_t p : s->selected[d - 1]) {
                    if (s->nodes[p].n_children < 0) all_expanded = false;
                    group_of(s, p, group);
                    members.insert(members.end(), group.begin(), group.end());
                }
            }
            members.erase(std::remove_if(members.begin(), members.end(),
                                         [s](int32_t x) { return s->nodes[x].state == kPruned; }),
                          members.end());
            const std::vector<int32_t> perfect = perfect_by_arrival(s, members);
            if (static_cast<int32_t>(perfect.size()) >= s->k) {  // rule 2
                decide(s, d, std::vector<int32_t>(perfect.begin(), perfect.begin() + s->k));
                changed = true;
                break;
            }
            if (rank_prune(s, members)) {  // rule 1
                changed = true;
                break;
            }
            bool all_scored = all_expanded;
            for (int32_t x : members) all_scored = all_scored && has_score(s->nodes[x]);
            if (all_scored) {
                std::vector<int32_t> ranked = members;
                std::sort(ranked.begin(), ranked.end(), [s](int32_t a, int32_t b) {
                    const Node &na = s->nodes[a], &nb = s->nodes[b];
                    return na.score != nb.score ? na.score > nb.score : na.arrival < nb.arrival;
                });
                ranked.resize(std::min<size_t>(ranked.size(), static_cast<size_t>(s->k)));
                decide(s, d, std::move(ranked));
                changed = true;
                break;
            }
        }
    }
}

bool group_complete(const tkv_search* s, int32_t parent) {
    std::vector<int32_t> g;
    group_of(s, parent, g);
    for (int32_t x : g)
        if (s->nodes[x].state == kGenerating) return false;
    return true;
}

bool should_flush(const tkv_search* s) {
    if (s->queue.empty()) return false;
    if (s->queued_tokens > s->threshold) return true;
    for (int32_t x : s->queue)
        if (s->nodes[x].deferrals >= s->max_deferrals) return true;
    for (int32_t x : s->queue)
        if (group_complete(s, s->nodes[x].parent)) return true;
    return false;
}

int check_node(const tkv_search* s, int32_t x, const char* fn) {
    if (x < 0 || x >= static_cast<int32_t>(s->nodes.size()))
        return set_error(TKV_EINVAL, "%s: no candidate %d (%zu exist)", fn, x, s->nodes.size());
    return TKV_OK;
}

}  // namespace

TKV_EXPORT int tkv_search_create(int32_t k, int32_t max_nodes, int32_t token_threshold, int32_t max_deferrals,
                                 tkv_search** out) {
    tkv::clear_error();
    if (!out) return set_error(TKV_EINVAL, "tkv_search_create: out is NULL");
    *out = nullptr;
    if (k < 1 || max_nodes < 1 || token_threshold < 0 || max_deferrals < 0)
        return set_error(TKV_EINVAL, "tkv_search_create: need k >= 1, max_nodes >= 1, threshold >= 0, max_deferrals >= 0 "
                                     "(got %d, %d, %d, %d)", k, max_nodes, token_threshold, max_deferrals);
    tkv_search* s = new (std::nothrow) tkv_search();
    if (!s) return set_error(TKV_ENOMEM, "tkv_search_create: host allocation failed");
    s->k = k;
    s->max_nodes = max_nodes;
    s->threshold = token_threshold;
    s->max_deferrals = max_deferrals;
    *out = s;
    return TKV_OK;
}

TKV_EXPORT void tkv_search_destroy(tkv_search* s) { delete s; }

TKV_EXPORT int tkv_search_expand(tkv_search* s, int32_t parent, int32_t n, int32_t* first_out) {
    tkv::clear_error();
    if (!s || !first_out) return set_error(TKV_EINVAL, "tkv_search_expand: NULL pointer");
    if (n < 0) return set_error(TKV_EINVAL, "tkv_search_expand: n = %d < 0", n);
    int32_t depth = 0;
    if (parent == -1) {
        if (s->n_roots >= 0) return set_error(TKV_EINVAL, "tkv_search_expand: the roots already exist");
    } else {
        if (int e = check_node(s, parent, "tkv_search_expand")) return e;
        const Node& p = s->nodes[parent];
        if (p.state == kPruned) return set_error(TKV_ENOSEQ, "tkv_search_expand: candidate %d is pruned", parent);
        if (!has_score(p))
            return set_error(TKV_EINVAL, "tkv_search_expand: candidate %d has no score yet (state %d)", parent, p.state);
        if (p.n_children >= 0) return set_error(TKV_EINVAL, "tkv_search_expand: candidate %d already expanded", parent);
        depth = p.depth + 1;
    }
    if (static_cast<int64_t>(s->nodes.size()) + n > s->max_nodes)
        return set_error(TKV_ENOMEM, "tkv_search_expand: %zu + %d candidates exceed max_nodes %d", s->nodes.size(), n,
                         s->max_nodes);
    const int32_t first = static_cast<int32_t>(s->nodes.size());
    try {
        for (int32_t i = 0; i < n; ++i) {
            Node c;
            c.parent = parent;
            c.depth = depth;
            s->nodes.push_back(c);
        }
    } catch (...) {
        s->nodes.resize(first);
        return set_error(TKV_ENOMEM, "tkv_search_expand: host allocation failed");
    }
    if (parent == -1) {
        s->n_roots = n;
    } else {
        s->nodes[parent].first_child = first;
        s->nodes[parent].n_children = n;
    }
    *first_out = first;
    settle(s);  // an expansion can complete a round's membership
    return TKV_OK;
}

TKV_EXPORT int tkv_search_complete(tkv_search* s, int32_t node, int32_t n_tokens, int32_t* flush_out) {
    tkv::clear_error();
    if (!s || !flush_out) return set_error(TKV_EINVAL, "tkv_search_complete: NULL pointer");
    if (int e = check_node(s, node, "tkv_search_complete")) return e;
    Node& n = s->nodes[node];
    if (n.state == kPruned) return set_error(TKV_ENOSEQ, "tkv_search_complete: candidate %d is pruned", node);
    if (n.state != kGenerating)
        return set_error(TKV_EINVAL, "tkv_search_complete: candidate %d already completed its step", node);
    if (n_tokens < 1) return set_error(TKV_EINVAL, "tkv_search_complete: n_tokens = %d < 1", n_tokens);
    s->queue.push_back(node);
    n.state = kQueued;
    n.tokens = n_tokens;
    n.deferrals = 0;
    s->queued_tokens += n_tokens;
    *flush_out = should_flush(s) ? 1 : 0;
    return TKV_OK;
}

TKV_EXPORT int tkv_search_tick(tkv_search* s, int32_t* flush_out) {
    tkv::clear_error();
    if (!s || !flush_out) return set_error(TKV_EINVAL, "tkv_search_tick: NULL pointer");
    const bool f = should_flush(s);
    if (!f)
        for (int32_t x : s->queue) ++s->nodes[x].deferrals;
    *flush_out = f ? 1 : 0;
    return TKV_OK;
}

TKV_EXPORT int tkv_search_flush(tkv_search* s, int32_t* nodes_out, int32_t cap, int32_t* n_out) {
    tkv::clear_error();
    if (!s || !n_out || (cap > 0 && !nodes_out)) return set_error(TKV_EINVAL, "tkv_search_flush: NULL pointer");
    const int32_t n = static_cast<int32_t>(s->queue.size());
    *n_out = n;
    if (cap < n) return set_error(TKV_ECAP, "tkv_search_flush: cap %d < %d queued", cap, n);
    for (int32_t i = 0; i < n; ++i) {
        nodes_out[i] = s->queue[i];
        s->nodes[s->queue[i]].state = kVerifying;
        s->nodes[s->queue[i]].flushed = true;
    }
    s->queue.clear();
    s->queued_tokens = 0;
    return TKV_OK;
}

TKV_EXPORT int tkv_search_score(tkv_search* s, int32_t n, const int32_t* nodes, const float* scores) {
    tkv::clear_error();
    if (!s || n < 0 || (n > 0 && (!nodes || !scores))) return set_error(TKV_EINVAL, "tkv_search_score: bad arguments");
    std::vector<uint8_t> seen(s->nodes.size(), 0);
    for (int32_t i = 0; i < n; ++i) {
        if (int e = check_node(s, nodes[i], "tkv_search_score")) return e;
        const Node& x = s->nodes[nodes[i]];
        if (!x.flushed || x.scored || seen[nodes[i]])
            return set_error(TKV_EINVAL, "tkv_search_score: candidate %d is not awaiting a score", nodes[i]);
        seen[nodes[i]] = 1;
        if (!(scores[i] >= 0.f && scores[i] <= 1.f))
            return set_error(TKV_EINVAL, "tkv_search_score: score %g of candidate %d is outside [0, 1]",
                             static_cast<double>(scores[i]), nodes[i]);
    }
    for (int32_t i = 0; i < n; ++i) {
        Node& x = s->nodes[nodes[i]];
        x.scored = true;
        if (x.state == kPruned) continue;  // pruned while its batch was verified: the score is moot
        x.state = kVerified;
        x.score = scores[i];
        x.arrival = s->n_arrivals++;
        settle(s);
    }
    return TKV_OK;
}

TKV_EXPORT int tkv_search_pruned(tkv_search* s, int32_t* nodes_out, int32_t cap, int32_t* n_out) {
    tkv::clear_error();
    if (!s || !n_out || (cap > 0 && !nodes_out)) return set_error(TKV_EINVAL, "tkv_search_pruned: NULL pointer");
    const int32_t n = static_cast<int32_t>(s->pending.size());
    *n_out = n;
    if (cap < n) return set_error(TKV_ECAP, "tkv_search_pruned: cap %d < %d pruned", cap, n);
    std::sort(s->pending.begin(), s->pending.end());
    std::copy(s->pending.begin(), s->pending.end(), nodes_out);
    s->pending.clear();
    return TKV_OK;
}

TKV_EXPORT int tkv_search_node(const tkv_search* s, int32_t node, int32_t* state_out, int32_t* parent_out,
                               int32_t* depth_out, float* score_out) {
    tkv::clear_error();
    if (!s || !state_out || !parent_out || !depth_out || !score_out)
        return set_error(TKV_EINVAL, "tkv_search_node: NULL pointer");
    if (int e = check_node(s, node, "tkv_search_node")) return e;
    const Node& n = s->nodes[node];
    *state_out = n.state;
    *parent_out = n.parent;
    *depth_out = n.depth;
    *score_out = n.scored && n.arrival >= 0 ? n.score : -1.f;
    return TKV_OK;
}

TKV_EXPORT int tkv_search_round(const tkv_search* s, int32_t depth, int32_t* selected_out, int32_t cap,
                                int32_t* n_out, int32_t* decided_out) {
    tkv::clear_error();
    if (!s || !n_out || !decided_out || (cap > 0 && !selected_out) || depth < 0)
        return set_error(TKV_EINVAL, "tkv_search_round: bad arguments");
    const bool known = depth < static_cast<int32_t>(s->decided.size()) && s->decided[depth];
    *decided_out = known ? 1 : 0;
    const int32_t n = known ? static_cast<int32_t>(s->selected[depth].size()) : 0;
    *n_out = n;
    if (cap < n) return set_error(TKV_ECAP, "tkv_search_round: cap %d < %d selected", cap, n);
    for (int32_t i = 0; i < n; ++i) selected_out[i] = s->selected[depth][i];
    return TKV_OK;
}

TKV_EXPORT int tkv_search_snapshot(const tkv_search* s, void* buf, size_t cap, size_t* used) {
    tkv::clear_error();
    if (!s || !used) return set_error(TKV_EINVAL, "tkv_search_snapshot: NULL pointer");
    std::vector<int32_t> w;
    w.push_back(s->k);
    w.push_back(s->threshold);
    w.push_back(s->max_deferrals);
    w.push_back(s->n_roots);
    w.push_back(static_cast<int32_t>(s->queued_tokens));
    w.push_back(static_cast<int32_t>(s->nodes.size()));
    for (const Node& n : s->nodes) {
        int32_t bits;
        std::memcpy(&bits, &n.score, 4);
        const int32_t words[] = {n.parent, n.depth, n.state, n.n_children, n.tokens, n.deferrals, n.arrival,
                                 n.arrival >= 0 ? bits : 0};
        w.insert(w.end(), std::begin(words), std::end(words));
    }
    w.push_back(static_cast<int32_t>(s->queue.size()));
    w.insert(w.end(), s->queue.begin(), s->queue.end());
    int32_t n_dec = 0;
    for (size_t d = 0; d < s->decided.size(); ++d)
        if (s->decided[d]) n_dec = static_cast<int32_t>(d) + 1;
    w.push_back(n_dec);
    for (int32_t d = 0; d < n_dec; ++d) {
        w.push_back(s->decided[d]);
        w.push_back(static_cast<int32_t>(s->selected[d].size()));
        w.insert(w.end(), s->selected[d].begin(), s->selected[d].end());
    }
    *used = w.size() * sizeof(int32_t);
    if (cap < *used) return set_error(TKV_ECAP, "tkv_search_snapshot: cap %zu < %zu bytes", cap, *used);
    std::memcpy(buf, w.data(), *used);
    return TKV_OK;
}
