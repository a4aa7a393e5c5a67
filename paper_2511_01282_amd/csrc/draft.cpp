// Host side of the drafting half of a ReSpec decoding step (include/respec_draft.h):
// the entropy-guided trigger (Section 3.2.1, Eq. 1-3), a suffix automaton over
// the context for retrieval, EMA-scored candidate selection (Section 3.3,
// Eq. 4-5), BuildDraftTree (Algorithm 1) and the per-sequence session that
// composes them in Algorithm 1's order.  Plain C++17; nothing here touches a GPU.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <string>
#include <unordered_map>
#include <utility>
#include <vector>

#include "../../include/respec_draft.h"

namespace {

// ---------------------------------------------------------------------------
// Transition table of the automaton: open addressing over (state, token) keys.
// Values index an edge array; each state also threads its edges in a list so
// that a clone can copy them.
// ---------------------------------------------------------------------------
class EdgeMap {
 public:
  EdgeMap() { rehash(1024); }

  int32_t find(int32_t state, int32_t tok) const {
    const uint64_t k = key(state, tok);
    for (size_t i = mix(k) & mask_;; i = (i + 1) & mask_) {
      if (keys_[i] == k) return vals_[i];
      if (keys_[i] == kEmpty) return -1;
    }
  }

  // Insert or overwrite.
  void put(int32_t state, int32_t tok, int32_t val) {
    if (2 * (used_ + 1) > keys_.size()) rehash(keys_.size() * 2);
    const uint64_t k = key(state, tok);
    size_t i = mix(k) & mask_;
    while (keys_[i] != kEmpty && keys_[i] != k) i = (i + 1) & mask_;
    if (keys_[i] == kEmpty) ++used_;
    keys_[i] = k;
    vals_[i] = val;
  }

 private:
  static constexpr uint64_t kEmpty = ~0ull;
  static uint64_t key(int32_t state, int32_t tok) { return ((uint64_t)(uint32_t)state << 32) | (uint32_t)tok; }
  // 64-bit finaliser (xor-shift / multiply rounds) so that consecutive states
  // and tokens spread over the table
  static uint64_t mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
  }
  void rehash(size_t cap) {
    std::vector<uint64_t> ok;
    std::vector<int32_t> ov;
    ok.swap(keys_);
    ov.swap(vals_);
    keys_.assign(cap, kEmpty);
    vals_.assign(cap, -1);
    mask_ = cap - 1;
    used_ = 0;
    for (size_t i = 0; i < ok.size(); ++i)
      if (ok[i] != kEmpty) {
        size_t j = mix(ok[i]) & mask_;
        while (keys_[j] != kEmpty) j = (j + 1) & mask_;
        keys_[j] = ok[i];
        vals_[j] = ov[i];
        ++used_;
      }
  }

  std::vector<uint64_t> keys_;
  std::vector<int32_t> vals_;
  size_t mask_ = 0, used_ = 0;
};

// Score table: open addressing over positions (>= 0), double values.
class ScoreMap {
 public:
  ScoreMap() { rehash(256); }
  double get(int32_t pos, double s0) const {
    for (size_t i = slot(pos);; i = (i + 1) & mask_) {
      if (keys_[i] == pos) return vals_[i];
      if (keys_[i] == kEmpty) return s0;
    }
  }
  void put(int32_t pos, double v) {
    if (2 * (used_ + 1) > keys_.size()) rehash(keys_.size() * 2);
    size_t i = slot(pos);
    while (keys_[i] != kEmpty && keys_[i] != pos) i = (i + 1) & mask_;
    if (keys_[i] == kEmpty) ++used_;
    keys_[i] = pos;
    vals_[i] = v;
  }
  size_t size() const { return used_; }

 private:
  static constexpr int32_t kEmpty = -1;
  size_t slot(int32_t pos) const { return ((uint32_t)pos * 0x9E3779B1u) & mask_; }
  void rehash(size_t cap) {
    std::vector<int32_t> ok;
    std::vector<double> ov;
    ok.swap(keys_);
    ov.swap(vals_);
    keys_.assign(cap, kEmpty);
    vals_.assign(cap, 0.0);
    mask_ = cap - 1;
    used_ = 0;
    for (size_t i = 0; i < ok.size(); ++i)
      if (ok[i] != kEmpty) put(ok[i], ov[i]);
  }
  std::vector<int32_t> keys_;
  std::vector<double> vals_;
  size_t mask_ = 0, used_ = 0;
};

constexpr double kNaN = __builtin_nan("");

}  // namespace

// ---------------------------------------------------------------------------
// Suffix automaton (Blumer et al.'s online construction).  Every state stands
// for a class of substrings with the same set of end positions; the suffix
// links form a tree in which the end positions of a state are the first end
// positions of the non-clone states of its subtree.  The link tree is kept as
// doubly linked child lists, so that the re-linking during a clone is O(1) and
// a retrieval visits only the subtree of the key's state.
// ---------------------------------------------------------------------------
struct respec_sam {
  struct Edge {
    int32_t tok, to, next;
  };
  std::vector<int32_t> len, link, firstpos, edge_head;
  std::vector<uint8_t> clone;
  std::vector<int32_t> child, next_sib, prev_sib;  // link tree
  std::vector<Edge> edges;
  EdgeMap trans;
  std::vector<int32_t> text;
  int32_t last = 0;

  respec_sam() { new_state(0, -1, false); }

  int32_t new_state(int32_t l, int32_t fpos, bool is_clone) {
    len.push_back(l);
    link.push_back(-1);
    firstpos.push_back(fpos);
    edge_head.push_back(-1);
    clone.push_back(is_clone);
    child.push_back(-1);
    next_sib.push_back(-1);
    prev_sib.push_back(-1);
    return (int32_t)len.size() - 1;
  }

  void set_edge(int32_t s, int32_t tok, int32_t to) {
    const int32_t e = trans.find(s, tok);
    if (e >= 0) {
      edges[e].to = to;
      return;
    }
    edges.push_back({tok, to, edge_head[s]});
    edge_head[s] = (int32_t)edges.size() - 1;
    trans.put(s, tok, edge_head[s]);
  }

  int32_t go(int32_t s, int32_t tok) const {
    const int32_t e = trans.find(s, tok);
    return e < 0 ? -1 : edges[e].to;
  }

  void set_link(int32_t v, int32_t u) {
    const int32_t old = link[v];
    if (old >= 0) {  // unlink v from old's children
      if (prev_sib[v] >= 0) next_sib[prev_sib[v]] = next_sib[v];
      else child[old] = next_sib[v];
      if (next_sib[v] >= 0) prev_sib[next_sib[v]] = prev_sib[v];
    }
    link[v] = u;
    prev_sib[v] = -1;
    next_sib[v] = child[u];
    if (child[u] >= 0) prev_sib[child[u]] = v;
    child[u] = v;
  }

  void extend(int32_t c) {
    const int32_t pos = (int32_t)text.size();
    text.push_back(c);
    const int32_t cur = new_state(len[last] + 1, pos, false);
    int32_t p = last;
    while (p >= 0 && go(p, c) < 0) {
      set_edge(p, c, cur);
      p = link[p];
    }
    if (p < 0) {
      set_link(cur, 0);
    } else {
      const int32_t q = go(p, c);
      if (len[p] + 1 == len[q]) {
        set_link(cur, q);
      } else {
        const int32_t cl = new_state(len[p] + 1, firstpos[q], true);
        for (int32_t e = edge_head[q]; e >= 0; e = edges[e].next) set_edge(cl, edges[e].tok, edges[e].to);
        set_link(cl, link[q]);
        while (p >= 0 && go(p, c) == q) {
          set_edge(p, c, cl);
          p = link[p];
        }
        set_link(q, cl);
        set_link(cur, cl);
      }
    }
    last = cur;
  }

  // State reached by reading key from the initial state, or -1.
  int32_t find(const int32_t* key, int32_t k) const {
    int32_t s = 0;
    for (int32_t i = 0; i < k && s >= 0; ++i) s = key[i] < 0 ? -1 : go(s, key[i]);
    return s;
  }

  // Retrieval positions of a key, ascending, kept per key and brought up to
  // date by scanning only the tokens appended since the last query (the
  // positions found earlier stay valid: the context only grows).  Keys that
  // repeat from step to step then cost the new tokens, not a walk of the
  // state's subtree (thousands of states for a frequent token).
  struct PosCache {
    std::vector<int32_t> asc;
    int64_t upto = 0;  // context length the list is complete for
  };
  static constexpr int kCacheMaxKey = 8;        // longer keys are not cached
  static constexpr size_t kCacheMaxEntries = 1024;
  mutable std::unordered_map<std::string, PosCache> pcache;
  mutable std::vector<int32_t> scratch;

  const std::vector<int32_t>& positions_asc(const int32_t* key, int32_t k) const {
    const int64_t n = (int64_t)text.size();
    if (k > kCacheMaxKey) {
      const int32_t st = find(key, k);
      scratch.clear();
      if (st > 0) positions(st, scratch);
      std::reverse(scratch.begin(), scratch.end());
      return scratch;
    }
    const std::string id(reinterpret_cast<const char*>(key), sizeof(int32_t) * (size_t)k);
    auto it = pcache.find(id);
    if (it == pcache.end()) {
      if (pcache.size() >= kCacheMaxEntries) pcache.clear();
      PosCache e;
      const int32_t st = find(key, k);
      if (st > 0) positions(st, e.asc);
      std::reverse(e.asc.begin(), e.asc.end());
      e.upto = n;
      return pcache.emplace(id, std::move(e)).first->second.asc;
    }
    PosCache& e = it->second;
    // new positions p (an occurrence ending at p with a following token): upto-1 <= p <= n-2
    for (int64_t p = std::max<int64_t>(e.upto - 1, k - 1); p <= n - 2; ++p) {
      bool m = true;
      for (int32_t i = 0; i < k && m; ++i) m = text[p - k + 1 + i] == key[i];
      if (m) e.asc.push_back((int32_t)p);
    }
    e.upto = n;
    return e.asc;
  }

  // End positions of state s with a following token, in decreasing order.
  void positions(int32_t s, std::vector<int32_t>& out) const {
    out.clear();
    const int32_t n = (int32_t)text.size();
    std::vector<int32_t> stack{s};
    while (!stack.empty()) {
      const int32_t v = stack.back();
      stack.pop_back();
      if (!clone[v] && firstpos[v] < n - 1) out.push_back(firstpos[v]);
      for (int32_t u = child[v]; u >= 0; u = next_sib[u]) stack.push_back(u);
    }
    std::sort(out.begin(), out.end(), std::greater<int32_t>());
  }
};

struct respec_scores {
  ScoreMap s;
  double get(int32_t pos, double s0) const { return pos < 0 ? s0 : s.get(pos, s0); }
};

struct respec_draft_session {
  respec_draft_params p;
  respec_sam sam;
  respec_scores scores;
  std::vector<float> entropy;  // entropy[i]: of the distribution that produced context token i
  // the last proposal, kept for commit
  bool have_proposal = false;
  respec_draft_result last;
  std::vector<int32_t> parent, token;
};

namespace {

bool trigger_params_ok(const respec_trigger_params* p) {
  return p->max_lookback >= 1 && isfinite(p->lambda_e) && isfinite(p->theta_entropy);
}
bool select_params_ok(const respec_select_params* p) {
  return p->alpha >= 0.f && p->alpha <= 1.f && isfinite(p->theta_score) && isfinite(p->s0) && p->n_select >= 1 &&
         p->n_select <= RESPEC_DRAFT_MAX_SELECT;
}
bool tree_params_ok(const respec_tree_params* p) {
  return p->max_draft_len >= 1 && p->max_nodes >= 2 && p->max_nodes <= RESPEC_MAX_NODES;
}

void trigger_eval(const float* e, int32_t n, const respec_trigger_params* p, respec_trigger_result* out) {
  respec_trigger_result r{0, (float)kNaN, (float)kNaN, 0};
  double c_min = 0, h_best = 0;
  for (int32_t k = 1; k <= p->max_lookback && k <= n; ++k) {
    bool finite = true;
    double sum = 0;
    for (int32_t i = n - k; i < n; ++i) {
      if (!isfinite(e[i])) finite = false;
      sum += (double)e[i];
    }
    if (!finite) break;  // every longer key holds the same token
    const double h = sum / k;
    const double c = h + (double)p->lambda_e / k;
    if (r.key_len == 0 || c < c_min) {
      c_min = c;
      h_best = h;
      r.key_len = k;
    }
  }
  if (r.key_len > 0) {
    r.h_min = (float)h_best;
    r.c_min = (float)c_min;
    r.fire = h_best <= (double)p->theta_entropy;
  }
  *out = r;
}

void select_positions(const respec_scores& sc, const int32_t* pos, int32_t n, const respec_select_params* p,
                      int32_t* sel, int32_t* n_sel) {
  std::vector<std::pair<double, int32_t>> kept;
  kept.reserve(n);
  const double s0 = p->s0, th = p->theta_score;
  for (int32_t i = 0; i < n; ++i) {
    const double s = sc.get(pos[i], s0);
    if (s >= th) kept.emplace_back(s, pos[i]);
  }
  const size_t m = std::min<size_t>(kept.size(), (size_t)p->n_select);
  std::partial_sort(kept.begin(), kept.begin() + m, kept.end(),
                    [](const std::pair<double, int32_t>& a, const std::pair<double, int32_t>& b) {
                      return a.first != b.first ? a.first > b.first : a.second > b.second;
                    });
  for (size_t i = 0; i < m; ++i) sel[i] = kept[i].second;
  *n_sel = (int32_t)m;
}

void ema_update(respec_scores& sc, const int32_t* sel, int32_t n_sel, int32_t winner, int32_t l_acc,
                const int32_t* l_draft, const respec_select_params* p) {
  const double a = (double)p->alpha;
  for (int32_t i = 0; i < n_sel; ++i) {
    const double r = i == winner ? (double)l_acc / (double)l_draft[i] : 0.0;
    const double s = sc.get(sel[i], (double)p->s0);
    sc.s.put(sel[i], (1.0 - a) * s + a * r);
  }
}

// Trie merge of the selected continuations (BuildDraftTree).
void build_tree(const respec_sam& sam, const int32_t* sel, int32_t n_sel, const respec_tree_params* p,
                int32_t* parent, int32_t* token, uint8_t* src, int32_t* n_nodes, int32_t* cand_end,
                int32_t* cand_len) {
  const int64_t n = (int64_t)sam.text.size();
  std::vector<int32_t> first_child(p->max_nodes, -1), next_sib(p->max_nodes, -1);
  int32_t cnt = 1;
  parent[0] = -1;
  token[0] = sam.text[n - 1];
  src[0] = RESPEC_SRC_MODEL;
  for (int32_t c = 0; c < n_sel; ++c) {
    int32_t node = 0, depth = 0;
    const int64_t end = std::min<int64_t>(n - 1, (int64_t)sel[c] + p->max_draft_len);
    for (int64_t t = (int64_t)sel[c] + 1; t <= end; ++t) {
      const int32_t tok = sam.text[t];
      int32_t ch = first_child[node];
      while (ch >= 0 && token[ch] != tok) ch = next_sib[ch];
      if (ch < 0) {
        if (cnt >= p->max_nodes) break;
        ch = cnt++;
        parent[ch] = node;
        token[ch] = tok;
        src[ch] = RESPEC_SRC_RETRIEVED;
        first_child[ch] = -1;
        // append at the end of node's child list (children in creation order)
        next_sib[ch] = -1;
        if (first_child[node] < 0) {
          first_child[node] = ch;
        } else {
          int32_t s = first_child[node];
          while (next_sib[s] >= 0) s = next_sib[s];
          next_sib[s] = ch;
        }
      }
      node = ch;
      ++depth;
    }
    cand_end[c] = node;
    cand_len[c] = depth;
  }
  *n_nodes = cnt;
}

}  // namespace

extern "C" {

respec_status respec_trigger_eval(const float* entropy, int32_t n, const respec_trigger_params* p,
                                  respec_trigger_result* out) {
  if (!p || !out || (n > 0 && !entropy)) return RESPEC_ERR_NULL;
  if (n < 0) return RESPEC_ERR_SHAPE;
  if (!trigger_params_ok(p)) return RESPEC_ERR_PARAM;
  trigger_eval(entropy, n, p, out);
  return RESPEC_OK;
}

respec_status respec_sam_create(respec_sam** out) {
  if (!out) return RESPEC_ERR_NULL;
  try {
    *out = new respec_sam();
  } catch (...) {
    return RESPEC_ERR_CAPACITY;
  }
  return RESPEC_OK;
}

void respec_sam_destroy(respec_sam* sam) { delete sam; }

respec_status respec_sam_extend(respec_sam* sam, const int32_t* tokens, int32_t n) {
  if (!sam || (n > 0 && !tokens)) return RESPEC_ERR_NULL;
  if (n < 0) return RESPEC_ERR_SHAPE;
  try {
    for (int32_t i = 0; i < n; ++i) {
      if (tokens[i] < 0) return RESPEC_ERR_TOKEN;
      sam->extend(tokens[i]);
    }
  } catch (...) {
    return RESPEC_ERR_CAPACITY;
  }
  return RESPEC_OK;
}

int64_t respec_sam_length(const respec_sam* sam) { return sam ? (int64_t)sam->text.size() : 0; }

respec_status respec_sam_text(const respec_sam* sam, int64_t start, int32_t n, int32_t* out) {
  if (!sam || (n > 0 && !out)) return RESPEC_ERR_NULL;
  if (start < 0 || n < 0 || start + n > (int64_t)sam->text.size()) return RESPEC_ERR_SHAPE;
  if (n > 0) memcpy(out, sam->text.data() + start, sizeof(int32_t) * (size_t)n);
  return RESPEC_OK;
}

respec_status respec_sam_positions(const respec_sam* sam, const int32_t* key, int32_t k, int32_t* pos_out,
                                   int32_t cap, int32_t* n_total) {
  if (!sam || !key || !n_total || (cap > 0 && !pos_out)) return RESPEC_ERR_NULL;
  if (k < 1 || cap < 0) return RESPEC_ERR_SHAPE;
  for (int32_t i = 0; i < k; ++i)
    if (key[i] < 0) return RESPEC_ERR_TOKEN;
  try {
    const std::vector<int32_t>& asc = sam->positions_asc(key, k);  // ascending
    const int32_t total = (int32_t)asc.size();
    const int32_t m = std::min<int32_t>(cap, total);
    for (int32_t j = 0; j < m; ++j) pos_out[j] = asc[total - 1 - j];  // most recent first
    *n_total = total;
  } catch (...) {
    return RESPEC_ERR_CAPACITY;
  }
  return RESPEC_OK;
}

respec_status respec_scores_create(respec_scores** out) {
  if (!out) return RESPEC_ERR_NULL;
  try {
    *out = new respec_scores();
  } catch (...) {
    return RESPEC_ERR_CAPACITY;
  }
  return RESPEC_OK;
}

void respec_scores_destroy(respec_scores* sc) { delete sc; }

double respec_scores_get(const respec_scores* sc, int32_t pos, double s0) { return sc ? sc->get(pos, s0) : s0; }

int64_t respec_scores_size(const respec_scores* sc) { return sc ? (int64_t)sc->s.size() : 0; }

respec_status respec_select(const respec_scores* sc, const int32_t* pos, int32_t n, const respec_select_params* p,
                            int32_t* sel_out, int32_t* n_sel) {
  if (!sc || !p || !sel_out || !n_sel || (n > 0 && !pos)) return RESPEC_ERR_NULL;
  if (n < 0) return RESPEC_ERR_SHAPE;
  for (int32_t i = 0; i < n; ++i)
    if (pos[i] < 0) return RESPEC_ERR_SHAPE;
  if (!select_params_ok(p)) return RESPEC_ERR_PARAM;
  try {
    select_positions(*sc, pos, n, p, sel_out, n_sel);
  } catch (...) {
    return RESPEC_ERR_CAPACITY;
  }
  return RESPEC_OK;
}

respec_status respec_scores_update(respec_scores* sc, const int32_t* sel, int32_t n_sel, int32_t winner,
                                   int32_t l_acc, const int32_t* l_draft, const respec_select_params* p) {
  if (!sc || !p || (n_sel > 0 && !sel) || (winner >= 0 && !l_draft)) return RESPEC_ERR_NULL;
  if (n_sel < 0 || n_sel > RESPEC_DRAFT_MAX_SELECT || winner < -1 || winner >= n_sel) return RESPEC_ERR_SHAPE;
  for (int32_t i = 0; i < n_sel; ++i)
    if (sel[i] < 0) return RESPEC_ERR_SHAPE;
  if (winner >= 0 && (l_draft[winner] < 1 || l_acc < 0 || l_acc > l_draft[winner])) return RESPEC_ERR_SHAPE;
  if (!select_params_ok(p)) return RESPEC_ERR_PARAM;
  try {
    ema_update(*sc, sel, n_sel, winner, l_acc, l_draft, p);
  } catch (...) {
    return RESPEC_ERR_CAPACITY;
  }
  return RESPEC_OK;
}

respec_status respec_build_tree(const respec_sam* sam, const int32_t* sel, int32_t n_sel, const respec_tree_params* p,
                                int32_t* parent, int32_t* token, uint8_t* src, int32_t* n_nodes, int32_t* cand_end,
                                int32_t* cand_len) {
  if (!sam || !p || !parent || !token || !src || !n_nodes || (n_sel > 0 && (!sel || !cand_end || !cand_len)))
    return RESPEC_ERR_NULL;
  if (!tree_params_ok(p)) return RESPEC_ERR_PARAM;
  const int64_t n = (int64_t)sam->text.size();
  if (n == 0 || n_sel < 0 || n_sel > RESPEC_DRAFT_MAX_SELECT) return RESPEC_ERR_SHAPE;
  for (int32_t c = 0; c < n_sel; ++c)
    if (sel[c] < 0 || sel[c] >= n) return RESPEC_ERR_SHAPE;
  try {
    build_tree(*sam, sel, n_sel, p, parent, token, src, n_nodes, cand_end, cand_len);
  } catch (...) {
    return RESPEC_ERR_CAPACITY;
  }
  return RESPEC_OK;
}

respec_status respec_draft_session_create(const respec_draft_params* p, respec_draft_session** out) {
  if (!p || !out) return RESPEC_ERR_NULL;
  if (!trigger_params_ok(&p->trigger) || !select_params_ok(&p->select) || !tree_params_ok(&p->tree))
    return RESPEC_ERR_PARAM;
  try {
    respec_draft_session* s = new respec_draft_session();
    s->p = *p;
    *out = s;
  } catch (...) {
    return RESPEC_ERR_CAPACITY;
  }
  return RESPEC_OK;
}

void respec_draft_session_destroy(respec_draft_session* s) { delete s; }

respec_status respec_draft_session_append(respec_draft_session* s, const int32_t* tokens, const float* entropy,
                                          int32_t n) {
  if (!s || (n > 0 && !tokens)) return RESPEC_ERR_NULL;
  if (n < 0) return RESPEC_ERR_SHAPE;
  for (int32_t i = 0; i < n; ++i)
    if (tokens[i] < 0) return RESPEC_ERR_TOKEN;
  try {
    for (int32_t i = 0; i < n; ++i) {
      s->sam.extend(tokens[i]);
      s->entropy.push_back(entropy ? entropy[i] : (float)kNaN);
    }
  } catch (...) {
    return RESPEC_ERR_CAPACITY;
  }
  return RESPEC_OK;
}

respec_status respec_draft_session_propose(respec_draft_session* s, int32_t* parent, int32_t* token, uint8_t* src,
                                           int32_t cap_nodes, respec_draft_result* out) {
  if (!s || !parent || !token || !src || !out) return RESPEC_ERR_NULL;
  const int32_t n = (int32_t)s->sam.text.size();
  if (n == 0 || cap_nodes < s->p.tree.max_nodes) return RESPEC_ERR_SHAPE;
  try {
    respec_draft_result r;
    memset(&r, 0, sizeof(r));
    // Step 1: the trigger over the entropies of the context's last l tokens
    const int32_t w = std::min(n, s->p.trigger.max_lookback);
    trigger_eval(s->entropy.data() + (n - w), w, &s->p.trigger, &r.trigger);
    static const std::vector<int32_t> kNone;
    const std::vector<int32_t>& pos =
        r.trigger.fire ? s->sam.positions_asc(s->sam.text.data() + (n - r.trigger.key_len), r.trigger.key_len)
                       : kNone;
    r.n_positions = (int32_t)pos.size();
    if (r.trigger.fire && !pos.empty()) {
      // Step 2: quality filtering, top-n selection (order-independent), BuildDraftTree
      select_positions(s->scores, pos.data(), (int32_t)pos.size(), &s->p.select, r.sel_pos, &r.n_selected);
      if (r.n_selected > 0) {
        build_tree(s->sam, r.sel_pos, r.n_selected, &s->p.tree, parent, token, src, &r.n_nodes, r.cand_end,
                   r.cand_len);
        r.retrieved = 1;
      }
    }
    if (!r.retrieved) {  // Step 3 belongs to the caller's drafter: hand back the root
      r.n_selected = 0;
      r.n_nodes = 1;
      parent[0] = -1;
      token[0] = s->sam.text[n - 1];
      src[0] = RESPEC_SRC_MODEL;
    }
    s->last = r;
    s->parent.assign(parent, parent + r.n_nodes);
    s->token.assign(token, token + r.n_nodes);
    s->have_proposal = true;
    *out = r;
  } catch (...) {
    return RESPEC_ERR_CAPACITY;
  }
  return RESPEC_OK;
}

respec_status respec_draft_session_commit(respec_draft_session* s, const int32_t* token, const int32_t* path,
                                          int32_t acc_len, int32_t bonus, const float* entropy) {
  if (!s || !token || !path || !entropy) return RESPEC_ERR_NULL;
  if (acc_len < 0 || bonus < 0) return acc_len < 0 ? RESPEC_ERR_SHAPE : RESPEC_ERR_TOKEN;
  for (int32_t j = 0; j <= acc_len; ++j)
    if (path[j] < 0) return RESPEC_ERR_SHAPE;
  for (int32_t j = 1; j <= acc_len; ++j)
    if (token[path[j]] < 0) return RESPEC_ERR_TOKEN;
  const bool retrieved = s->have_proposal && s->last.retrieved;
  if (retrieved) {
    const int32_t nn = (int32_t)s->parent.size();
    if (path[0] != 0) return RESPEC_ERR_TREE;
    for (int32_t j = 1; j <= acc_len; ++j)
      if (path[j] >= nn || s->parent[path[j]] != path[j - 1]) return RESPEC_ERR_TREE;
  }
  try {
    if (retrieved) {
      // winner: the first selected candidate whose chain holds the last accepted node
      const respec_draft_result& r = s->last;
      const int32_t tip = path[acc_len];
      int32_t winner = -1;
      for (int32_t c = 0; c < r.n_selected && winner < 0; ++c)
        for (int32_t v = r.cand_end[c]; v >= 0; v = s->parent[v])
          if (v == tip) {
            winner = c;
            break;
          }
      if (winner >= 0 && r.cand_len[winner] < 1) winner = -1;  // only the root: nothing drafted
      ema_update(s->scores, r.sel_pos, r.n_selected, winner, acc_len, r.cand_len, &s->p.select);
    }
    for (int32_t j = 1; j <= acc_len; ++j) {
      s->sam.extend(token[path[j]]);
      s->entropy.push_back(entropy[path[j - 1]]);
    }
    s->sam.extend(bonus);
    s->entropy.push_back(entropy[path[acc_len]]);
    s->have_proposal = false;
  } catch (...) {
    return RESPEC_ERR_CAPACITY;
  }
  return RESPEC_OK;
}

const respec_sam* respec_draft_session_sam(const respec_draft_session* s) { return s ? &s->sam : nullptr; }
const respec_scores* respec_draft_session_scores(const respec_draft_session* s) { return s ? &s->scores : nullptr; }

}  // extern "C"
