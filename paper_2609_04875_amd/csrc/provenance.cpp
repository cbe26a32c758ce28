// Forget front-end: the provenance graph of Section 3.4 (a), the influence set
// of Lemma 2, checkpoint selection (Section 3.4 (b); Algorithm 1, the steps
// before the restore) and the Corollary 1 counts.  Host code.
//
// Layout.  Per artifact: type (int8), turn (int32), span end (int64), a
// committed flag, and CSR ranges into one parent array (int32 ids) and one
// source-id array (int64).  Because artifacts arrive in turn order and a parent
// always precedes its child, ids are a topological order of G and turns are
// sorted; prefix arrays over ids then answer "KV length after turn b" (running
// max of span ends), "artifacts before tau" and "committed side effects from
// tau on" by binary search.  A hash index maps each source id to the
// artifacts that introduce it.
//
// Children are kept as per-parent linked lists over the edge array (head per
// artifact, next per edge), filled at append time.  Taint closure: a
// breadth-first walk from the seeds over those lists, so a query costs the
// closure's own artifacts and out-edges, not the graph after the seeds; the
// ids found are sorted at the end.
#include <algorithm>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <iterator>
#include <new>
#include <unordered_map>
#include <vector>

#include "internal.h"
#include "pgsr.h"

struct pgsr_graph {
  int64_t cap_art = 0, cap_edge = 0, cap_src = 0;
  std::vector<int8_t> type;
  std::vector<int32_t> turn;
  std::vector<int64_t> span_end;
  std::vector<int64_t> kv_after;      // running max of span_end over ids 0..i
  std::vector<int64_t> committed_before;  // committed artifacts among ids 0..i-1 (size n+1)
  std::vector<int64_t> par_off;       // size n+1
  std::vector<int32_t> par;
  std::vector<int32_t> child_head;    // per artifact: last edge naming it as parent, -1 if none
  std::vector<int32_t> edge_next;     // per edge: previous edge of the same parent, -1 at the end
  std::vector<int32_t> edge_child;    // per edge: the child
  std::vector<int64_t> src_off;       // size n+1
  std::vector<int64_t> src;
  std::unordered_map<int64_t, std::vector<int32_t>> entries;   // source id -> artifacts
  mutable std::vector<uint8_t> mark;  // closure scratch, all zero between calls
};

struct pgsr_ckpt_store {
  struct Rec {
    int64_t boundary, token_offset, seq, env_snapshot, manifest;
  };
  int64_t cap = 0;
  std::vector<Rec> recs;
  std::vector<std::pair<int64_t, int64_t>> order;   // (boundary, index), ascending
};

namespace {

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  pgsr::set_error(buf);
  return code;
}

int ok() {
  pgsr::clear_error();
  return PGSR_OK;
}

// Copy n ascending ids to out if it fits (all-or-nothing).
int emit(const std::vector<int64_t>& ids, int64_t* out, int64_t capacity, int64_t* n_out) {
  if (n_out) *n_out = (int64_t)ids.size();
  if (out == nullptr && capacity == 0) return ok();
  if (out == nullptr || capacity < (int64_t)ids.size())
    return fail(PGSR_ERANGE, "output holds %lld ids, %lld needed", (long long)capacity,
                (long long)ids.size());
  std::copy(ids.begin(), ids.end(), out);
  return ok();
}

int64_t last_turn(const pgsr_graph* g) { return g->turn.empty() ? 0 : g->turn.back(); }

// Artifacts with turn < t: the first id whose turn is >= t.
int64_t count_before_turn(const pgsr_graph* g, int64_t t) {
  return std::lower_bound(g->turn.begin(), g->turn.end(), t,
                          [](int32_t a, int64_t b) { return (int64_t)a < b; }) -
         g->turn.begin();
}

int64_t kv_length_after(const pgsr_graph* g, int64_t b) {
  const int64_t n = count_before_turn(g, b + 1);   // artifacts of turns <= b
  return n == 0 ? 0 : g->kv_after[n - 1];
}

void closure(const pgsr_graph* g, const std::vector<int64_t>& seeds, std::vector<int64_t>& out) {
  out.clear();
  for (int64_t s : seeds)
    if (!g->mark[s]) {
      g->mark[s] = 1;
      out.push_back(s);
    }
  for (size_t i = 0; i < out.size(); ++i)
    for (int32_t e = g->child_head[out[i]]; e >= 0; e = g->edge_next[e]) {
      const int32_t c = g->edge_child[e];
      if (!g->mark[c]) {
        g->mark[c] = 1;
        out.push_back(c);
      }
    }
  for (int64_t a : out) g->mark[a] = 0;
  std::sort(out.begin(), out.end());
}

}  // namespace

extern "C" {

int pgsr_graph_create(int64_t max_artifacts, int64_t max_edges, int64_t max_sources,
                      pgsr_graph** out) {
  if (!out) return fail(PGSR_EINVAL, "out is NULL");
  *out = nullptr;
  if (max_artifacts < 0 || max_edges < 0 || max_sources < 0)
    return fail(PGSR_EINVAL, "negative capacity");
  if (max_artifacts >= INT32_MAX || max_edges >= INT32_MAX)
    return fail(PGSR_EINVAL, "at most 2^31 - 2 artifacts and edges");
  pgsr_graph* g = new (std::nothrow) pgsr_graph;
  if (!g) return fail(PGSR_ENOMEM, "host allocation failed");
  try {
    g->cap_art = max_artifacts;
    g->cap_edge = max_edges;
    g->cap_src = max_sources;
    g->type.reserve(max_artifacts);
    g->turn.reserve(max_artifacts);
    g->span_end.reserve(max_artifacts);
    g->kv_after.reserve(max_artifacts);
    g->committed_before.reserve(max_artifacts + 1);
    g->committed_before.push_back(0);
    g->par_off.reserve(max_artifacts + 1);
    g->par_off.push_back(0);
    g->src_off.reserve(max_artifacts + 1);
    g->src_off.push_back(0);
    g->par.reserve(max_edges);
    g->child_head.reserve(max_artifacts);
    g->edge_next.reserve(max_edges);
    g->edge_child.reserve(max_edges);
    g->src.reserve(max_sources);
    g->mark.assign(max_artifacts, 0);
  } catch (const std::bad_alloc&) {
    delete g;
    return fail(PGSR_ENOMEM, "host allocation failed");
  }
  *out = g;
  return ok();
}

int pgsr_graph_destroy(pgsr_graph* g) {
  delete g;
  return ok();
}

int pgsr_graph_append(pgsr_graph* g, int64_t n, const int32_t* types, const int32_t* turns,
                      const int64_t* span_begin, const int64_t* span_end,
                      const int64_t* parent_off, const int64_t* parents,
                      const int64_t* source_off, const int64_t* sources,
                      const uint8_t* committed, int64_t* first_id) {
  if (!g) return fail(PGSR_EINVAL, "graph is NULL");
  if (n < 0) return fail(PGSR_EINVAL, "negative count");
  if (n > 0 && (!types || !turns || !span_begin || !span_end || !parent_off || !source_off))
    return fail(PGSR_EINVAL, "NULL record array");
  const int64_t base = (int64_t)g->turn.size();
  if (n > 0 && (parent_off[0] != 0 || source_off[0] != 0))
    return fail(PGSR_EINVAL, "offsets must start at 0");
  // validate the whole batch first
  int64_t prev_turn = last_turn(g);
  for (int64_t i = 0; i < n; ++i) {
    const int64_t id = base + i;
    if (types[i] < 0 || types[i] > PGSR_ART_SUMMARY)
      return fail(PGSR_EINVAL, "artifact %lld: unknown type %d", (long long)id, types[i]);
    if (turns[i] < 1) return fail(PGSR_EINVAL, "artifact %lld: turns start at 1", (long long)id);
    if (turns[i] < prev_turn)
      return fail(PGSR_EINVAL, "artifact %lld: turn %d after turn %lld (artifacts arrive in turn order)",
                  (long long)id, turns[i], (long long)prev_turn);
    prev_turn = turns[i];
    if (span_begin[i] < 0 || span_end[i] < span_begin[i])
      return fail(PGSR_EINVAL, "artifact %lld: bad token span", (long long)id);
    if (parent_off[i + 1] < parent_off[i] || source_off[i + 1] < source_off[i])
      return fail(PGSR_EINVAL, "artifact %lld: decreasing offsets", (long long)id);
    if (committed && committed[i] > 1)
      return fail(PGSR_EINVAL, "artifact %lld: committed must be 0 or 1", (long long)id);
    for (int64_t e = parent_off[i]; e < parent_off[i + 1]; ++e) {
      const int64_t p = parents ? parents[e] : -1;
      if (p < 0 || p >= id)
        return fail(PGSR_EINVAL, "artifact %lld: parent %lld does not exist", (long long)id, (long long)p);
      const int32_t pt = p < base ? g->turn[p] : turns[p - base];
      if (pt > turns[i])
        return fail(PGSR_EINVAL, "artifact %lld: parent %lld is of a later turn", (long long)id,
                    (long long)p);
    }
    if (source_off[i + 1] > source_off[i] && !sources)
      return fail(PGSR_EINVAL, "sources is NULL");
  }
  const int64_t n_edges = n > 0 ? parent_off[n] : 0, n_src = n > 0 ? source_off[n] : 0;
  if (base + n > g->cap_art || (int64_t)g->par.size() + n_edges > g->cap_edge ||
      (int64_t)g->src.size() + n_src > g->cap_src)
    return fail(PGSR_ENOMEM, "graph capacity exceeded");
  try {
    for (int64_t i = 0; i < n; ++i) {
      const int64_t id = base + i;
      for (int64_t e = source_off[i]; e < source_off[i + 1]; ++e) {
        auto& v = g->entries[sources[e]];
        if (v.empty() || v.back() != (int32_t)id) v.push_back((int32_t)id);
      }
    }
  } catch (const std::bad_alloc&) {
    // take this batch's ids back out of the index (they are the newest entries)
    for (auto it = g->entries.begin(); it != g->entries.end();) {
      while (!it->second.empty() && it->second.back() >= base) it->second.pop_back();
      it = it->second.empty() ? g->entries.erase(it) : std::next(it);
    }
    return fail(PGSR_ENOMEM, "host allocation failed");
  }
  for (int64_t i = 0; i < n; ++i) {
    const int64_t id = base + i;
    g->type.push_back((int8_t)types[i]);
    g->turn.push_back(turns[i]);
    g->span_end.push_back(span_end[i]);
    g->kv_after.push_back(g->kv_after.empty() ? span_end[i] : std::max(g->kv_after.back(), span_end[i]));
    g->committed_before.push_back(g->committed_before.back() + (committed && committed[i] ? 1 : 0));
    g->child_head.push_back(-1);
    for (int64_t e = parent_off[i]; e < parent_off[i + 1]; ++e) {
      const int32_t p = (int32_t)parents[e], edge = (int32_t)g->par.size();
      g->par.push_back(p);
      g->edge_child.push_back((int32_t)id);
      g->edge_next.push_back(g->child_head[p]);
      g->child_head[p] = edge;
    }
    g->par_off.push_back((int64_t)g->par.size());
    for (int64_t e = source_off[i]; e < source_off[i + 1]; ++e) g->src.push_back(sources[e]);
    g->src_off.push_back((int64_t)g->src.size());
  }
  if (first_id) *first_id = base;
  return ok();
}

int pgsr_graph_size(const pgsr_graph* g, int64_t* n_out) {
  if (!g || !n_out) return fail(PGSR_EINVAL, "NULL argument");
  *n_out = (int64_t)g->turn.size();
  return ok();
}

int pgsr_graph_session_length(const pgsr_graph* g, int64_t* T_out) {
  if (!g || !T_out) return fail(PGSR_EINVAL, "NULL argument");
  *T_out = last_turn(g);
  return ok();
}

int pgsr_graph_kv_length_after(const pgsr_graph* g, int64_t b, int64_t* len_out) {
  if (!g || !len_out) return fail(PGSR_EINVAL, "NULL argument");
  if (b < 0) return fail(PGSR_EINVAL, "negative boundary");
  *len_out = kv_length_after(g, b);
  return ok();
}

int pgsr_graph_locate_source(const pgsr_graph* g, int64_t z, int64_t* out, int64_t capacity,
                             int64_t* n_out) {
  if (!g) return fail(PGSR_EINVAL, "graph is NULL");
  if (capacity < 0) return fail(PGSR_EINVAL, "negative capacity");
  std::vector<int64_t> ids;
  const auto it = g->entries.find(z);
  if (it != g->entries.end()) ids.assign(it->second.begin(), it->second.end());
  return emit(ids, out, capacity, n_out);
}

int pgsr_graph_taint_closure(const pgsr_graph* g, const int64_t* seeds, int64_t n_seeds,
                             int64_t* out, int64_t capacity, int64_t* n_out) {
  if (!g) return fail(PGSR_EINVAL, "graph is NULL");
  if (n_seeds < 0 || capacity < 0 || (n_seeds > 0 && !seeds))
    return fail(PGSR_EINVAL, "bad seed list");
  const int64_t n = (int64_t)g->turn.size();
  std::vector<int64_t> sv(seeds, seeds + n_seeds), ids;
  for (int64_t s : sv)
    if (s < 0 || s >= n) return fail(PGSR_EINVAL, "seed %lld does not exist", (long long)s);
  closure(g, sv, ids);
  return emit(ids, out, capacity, n_out);
}

int pgsr_graph_policy_boundaries(const pgsr_graph* g, int32_t policy, int64_t k, int64_t* out,
                                 int64_t capacity, int64_t* n_out) {
  if (!g) return fail(PGSR_EINVAL, "graph is NULL");
  if (capacity < 0) return fail(PGSR_EINVAL, "negative capacity");
  const int64_t T = last_turn(g);
  std::vector<int64_t> b;
  switch (policy) {
    case PGSR_POLICY_EVERY_TURN:
      for (int64_t t = 0; t < T; ++t) b.push_back(t);
      break;
    case PGSR_POLICY_SESSION_START:
      b.push_back(0);
      break;
    case PGSR_POLICY_BEFORE_INJECTION: {
      b.push_back(0);
      const int64_t n = (int64_t)g->turn.size();
      for (int64_t a = 0; a < n; ++a)       // turns ascend, so boundaries come out sorted
        if (g->src_off[a + 1] > g->src_off[a] && g->turn[a] - 1 > b.back()) b.push_back(g->turn[a] - 1);
      break;
    }
    case PGSR_POLICY_EVERY_K:
      if (k < 1) return fail(PGSR_EINVAL, "k must be >= 1");
      for (int64_t t = 0; t < T; t += k) b.push_back(t);
      break;
    default:
      return fail(PGSR_EINVAL, "unknown policy %d", policy);
  }
  return emit(b, out, capacity, n_out);
}

int pgsr_ckpt_create(int64_t capacity, pgsr_ckpt_store** out) {
  if (!out) return fail(PGSR_EINVAL, "out is NULL");
  *out = nullptr;
  if (capacity < 0) return fail(PGSR_EINVAL, "negative capacity");
  pgsr_ckpt_store* s = new (std::nothrow) pgsr_ckpt_store;
  if (!s) return fail(PGSR_ENOMEM, "host allocation failed");
  try {
    s->cap = capacity;
    s->recs.reserve(capacity);
    s->order.reserve(capacity);
  } catch (const std::bad_alloc&) {
    delete s;
    return fail(PGSR_ENOMEM, "host allocation failed");
  }
  *out = s;
  return ok();
}

int pgsr_ckpt_destroy(pgsr_ckpt_store* s) {
  delete s;
  return ok();
}

int pgsr_ckpt_register(pgsr_ckpt_store* s, int64_t boundary, int64_t token_offset, int64_t seq,
                       int64_t env_snapshot, int64_t manifest) {
  if (!s) return fail(PGSR_EINVAL, "store is NULL");
  if (boundary < 0 || token_offset < 0) return fail(PGSR_EINVAL, "negative boundary or offset");
  if ((int64_t)s->recs.size() >= s->cap) return fail(PGSR_ENOMEM, "checkpoint store is full");
  const int64_t idx = (int64_t)s->recs.size();
  s->recs.push_back({boundary, token_offset, seq, env_snapshot, manifest});
  const std::pair<int64_t, int64_t> key{boundary, idx};
  s->order.insert(std::upper_bound(s->order.begin(), s->order.end(), key), key);
  return ok();
}

int pgsr_ckpt_count(const pgsr_ckpt_store* s, int64_t* n_out) {
  if (!s || !n_out) return fail(PGSR_EINVAL, "NULL argument");
  *n_out = (int64_t)s->recs.size();
  return ok();
}

int pgsr_forget_plan_query(const pgsr_graph* g, const pgsr_ckpt_store* s, int64_t z,
                           int64_t* closure_out, int64_t capacity, pgsr_forget_plan* plan) {
  if (!g || !s || !plan) return fail(PGSR_EINVAL, "NULL argument");
  if (capacity < 0) return fail(PGSR_EINVAL, "negative capacity");
  const auto it = g->entries.find(z);
  if (it == g->entries.end()) return fail(PGSR_ENOENT, "target %lld never entered", (long long)z);
  std::vector<int64_t> seeds(it->second.begin(), it->second.end());
  const int64_t tau = g->turn[seeds.front()];   // ids ascend, turns ascend with them
  // c* = the largest boundary below tau; among equals the last registered
  const auto pos = std::lower_bound(s->order.begin(), s->order.end(),
                                    std::pair<int64_t, int64_t>{tau, INT64_MIN});
  if (pos == s->order.begin())
    return fail(PGSR_ENOENT, "no checkpoint below tau = %lld", (long long)tau);
  const int64_t ci = std::prev(pos)->second;
  const auto& c = s->recs[ci];
  std::vector<int64_t> ids;
  closure(g, seeds, ids);
  const int64_t T = last_turn(g), n = (int64_t)g->turn.size();
  const int64_t clean = count_before_turn(g, tau);
  pgsr_forget_plan p;
  p.tau = tau;
  p.checkpoint = ci;
  p.boundary = c.boundary;
  p.crop_len = c.token_offset;
  p.seq = c.seq;
  p.env_snapshot = c.env_snapshot;
  p.manifest = c.manifest;
  p.replay_transitions = T - c.boundary;
  p.minimal_transitions = T - tau + 1;
  p.n_sources = (int64_t)seeds.size();
  p.closure_size = (int64_t)ids.size();
  p.clean_artifacts = clean;
  p.committed_after_tau = g->committed_before[n] - g->committed_before[clean];
  *plan = p;
  if (closure_out == nullptr) return ok();
  int64_t unused;
  return emit(ids, closure_out, capacity, &unused);
}

}  // extern "C"
