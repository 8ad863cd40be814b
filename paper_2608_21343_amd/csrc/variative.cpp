// Host compiler of the case-insensitive variative BPE graph (Sec. II-A,
// Fig. 1c and 1e, Eq. (1)) into the same arena image as tb_compile_graphs.
//
// A phrase is a character string. Its lowercased characters form a chain, and
// every vocabulary piece whose lowercased string spans a contiguous segment of
// the chain is an arc over that segment (single-character pieces give the
// chain itself, longer pieces the merged arcs). Merging all phrases of a list
// gives a character trie of nodes with these arcs on top: a DAG, because arcs
// of different lengths reach the same node, plus character-level suffix
// links. Arcs are labelled by piece class (all pieces with one lowercased
// string), so one arc accepts every cased spelling.
//
// Scores (Eq. (1)): each phrase's greedy tokenization (longest match from the
// left over the lowercased pieces) is its scoring backbone; backbone token k,
// with score w and m_k characters, gives its i-th character the share
// w * exp((i+1)^tau) / sum_j exp((j+1)^tau). P(node) is the running sum of
// shares along a phrase (the largest over the phrases through the node), and
// the potentials follow the reading of the class graph with the token count
// replaced by P:
//   commit: phi(x) = alpha*(P(x) - P(e(x))), e(x) = deepest phrase end on x's
//           path (x included, else the root);
//           E(x) = alpha*(P(x) - P(e(parent x)) + bonus) if x ends a phrase,
//                  alpha*bonus if a proper suffix does, else 0;
//   pure:   phi(x) = alpha*P(x), E(x) = alpha*bonus if x or a suffix ends one.
//
// Encoding for the step kernels, which walk tree-shaped records: every arc is
// a state standing for its target node, so a node reached by several arcs has
// several states, all with the node's potentials, the node's out-arcs as their
// children and the first arc into the node's longest proper suffix node as
// their suffix link. Nodes are expanded by increasing length, nodes of one
// length in the order of their first arc; expanding a node numbers its
// out-arcs consecutively in ascending class order (root = state 0). Suffix
// links therefore need not point to smaller ids; they still strictly shorten
// the node's string, so every suffix chain ends at the root.

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <map>
#include <thread>
#include <unordered_map>

#include "internal.hpp"

namespace tbias {

namespace {

// Lowercased pieces: a trie over characters whose terminal nodes carry the
// piece class (the smallest token id with that lowercased string).
struct PieceTrie {
  std::vector<std::map<int32_t, int32_t>> next{1};
  std::vector<int32_t> cls{-1};
  int32_t child(int32_t u, int32_t ch) const {
    auto it = next[u].find(ch);
    return it == next[u].end() ? -1 : it->second;
  }
};

struct CharTrie {
  std::vector<int32_t> parent{-1}, depth{0}, ch{-1};
  std::vector<std::map<int32_t, int32_t>> next{1};
  std::vector<char> fin{0};
  int32_t child(int32_t u, int32_t c) const {
    auto it = next[u].find(c);
    return it == next[u].end() ? -1 : it->second;
  }
  int32_t add(int32_t u, int32_t c) {
    int32_t v = child(u, c);
    if (v >= 0) return v;
    v = (int32_t)parent.size();
    parent.push_back(u);
    depth.push_back(depth[u] + 1);
    ch.push_back(c);
    next.emplace_back();
    fin.push_back(0);
    next[u][c] = v;
    return v;
  }
};

int compile_variative_model(const std::vector<std::vector<int32_t>>& phrases,
                            const PieceTrie& pt, const int32_t* class_map, int32_t V, double w,
                            double bonus, double alpha, double tau, int32_t semantics,
                            ModelGraph* out) {
  // 1. character trie of the (lowercased, deduplicated) phrases
  CharTrie tr;
  for (const auto& p : phrases) {
    int32_t u = 0;
    for (int32_t c : p) {
      if (pt.child(0, c) < 0 || pt.cls[pt.child(0, c)] < 0)
        return fail(TB_ERANGE, "character " + std::to_string(c) +
                                   " is not a single-character piece of the vocabulary");
      u = tr.add(u, c);
    }
    tr.fin[u] = 1;
  }
  const int32_t nn = (int32_t)tr.parent.size();

  // 2. backbone potentials: running sums of the Eq. (1) shares along every
  //    phrase, in the phrase's character order; a node keeps the largest
  std::vector<double> P(nn, -HUGE_VAL);
  P[0] = 0.0;
  for (const auto& p : phrases) {
    const int32_t L = (int32_t)p.size();
    double acc = 0.0;
    int32_t u = 0, i = 0;
    while (i < L) {
      int32_t best = 0;  // longest piece starting at i
      for (int32_t q = 0, j = i; j < L; ++j) {
        q = pt.child(q, p[j]);
        if (q < 0) break;
        if (pt.cls[q] >= 0) best = j - i + 1;
      }
      const int32_t m = best;  // >= 1: every character is a piece
      double den = 0.0;
      for (int32_t j = 0; j < m; ++j) den += std::exp(std::pow((double)(j + 1), tau));
      for (int32_t k = 0; k < m; ++k) {
        acc += w * std::exp(std::pow((double)(k + 1), tau)) / den;
        u = tr.child(u, p[i + k]);
        P[u] = std::max(P[u], acc);
      }
      i += m;
    }
  }

  // 3. character-level suffix links (longest proper suffix that is a node),
  //    breadth first over the trie
  std::vector<int32_t> clink(nn, 0), bfs;
  bfs.reserve(nn);
  bfs.push_back(0);
  for (size_t h = 0; h < bfs.size(); ++h) {
    const int32_t x = bfs[h];
    for (const auto& kv : tr.next[x]) {
      const int32_t y = kv.second, c = kv.first;
      if (x == 0) {
        clink[y] = 0;
      } else {
        int32_t f = clink[x];
        for (;;) {
          const int32_t z = tr.child(f, c);
          if (z >= 0) { clink[y] = z; break; }
          if (f == 0) { clink[y] = 0; break; }
          f = clink[f];
        }
      }
      bfs.push_back(y);
    }
  }

  // 4. out-arcs of every node: walk the piece trie along the phrase trie
  std::vector<std::vector<std::pair<int32_t, int32_t>>> arcs(nn);  // (class, target node)
  for (int32_t x = 0; x < nn; ++x) {
    // depth-first over common continuations
    std::vector<std::pair<int32_t, int32_t>> stack{{0, x}};  // (piece node, trie node)
    while (!stack.empty()) {
      const auto [q, u] = stack.back();
      stack.pop_back();
      for (const auto& kv : pt.next[q]) {
        const int32_t v = tr.child(u, kv.first);
        if (v < 0) continue;
        if (pt.cls[kv.second] >= 0) arcs[x].push_back({pt.cls[kv.second], v});
        stack.push_back({kv.second, v});
      }
    }
    std::sort(arcs[x].begin(), arcs[x].end());
  }

  // 5. numbering: nodes by depth, one depth in order of first arc
  std::vector<int32_t> rep(nn, -1), blk(nn, 0), target{0};
  rep[0] = 0;
  int32_t max_depth = 0;
  for (int32_t x = 0; x < nn; ++x) max_depth = std::max(max_depth, tr.depth[x]);
  std::vector<std::vector<int32_t>> level(max_depth + 1);
  level[0].push_back(0);
  int64_t n_states = 1;
  for (int32_t L = 0; L <= max_depth; ++L) {
    for (size_t h = 0; h < level[L].size(); ++h) {
      const int32_t x = level[L][h];
      blk[x] = (int32_t)n_states;
      for (const auto& a : arcs[x]) {
        const int32_t T = a.second;
        if (rep[T] < 0) {
          rep[T] = (int32_t)n_states;
          level[tr.depth[T]].push_back(T);
        }
        target.push_back(T);
        ++n_states;
        if (n_states > INT32_MAX / 2) return fail(TB_ERANGE, "too many arcs in one model");
      }
    }
  }
  for (int32_t x = 0; x < nn; ++x)
    if (rep[x] < 0) return fail(TB_ERANGE, "unreachable node (internal)");

  // 6. node potentials
  std::vector<int32_t> endn(nn, 0);          // deepest phrase end on the path (x included)
  std::vector<char> suf_final(nn, 0);        // a proper suffix ends a phrase
  std::vector<float> nphi(nn, 0.f), npsi(nn, 0.f);
  for (size_t h = 1; h < bfs.size(); ++h) {  // parents before children, links shallower
    const int32_t y = bfs[h], par = tr.parent[y], l = clink[y];
    endn[y] = tr.fin[y] ? y : endn[par];
    suf_final[y] = (l != 0) && (tr.fin[l] || suf_final[l]);
    double phi, E;
    if (semantics == TB_COMMIT) {
      phi = alpha * (P[y] - P[endn[y]]);
      if (tr.fin[y]) E = alpha * ((P[y] - P[endn[par]]) + bonus);
      else if (suf_final[y]) E = alpha * bonus;
      else E = 0.0;
    } else {
      phi = alpha * P[y];
      E = (tr.fin[y] || suf_final[y]) ? alpha * bonus : 0.0;
    }
    nphi[y] = (float)phi;
    npsi[y] = (float)(phi + E);
  }

  // 7. state arrays
  ModelGraph& g = *out;
  const int32_t n = (int32_t)n_states;
  g.n = n;
  g.first_child.assign(n, 0);
  g.n_child.assign(n, 0);
  g.link.assign(n, 0);
  g.label.assign(n, -1);
  g.phi.assign(n, 0.f);
  g.psi.assign(n, 0.f);
  g.max_depth = max_depth;
  for (int32_t x = 0; x < nn; ++x)
    for (size_t j = 0; j < arcs[x].size(); ++j) g.label[blk[x] + (int32_t)j] = arcs[x][j].first;
  for (int32_t s = 0; s < n; ++s) {
    const int32_t T = target[s];
    const int32_t nc = (int32_t)arcs[T].size();
    g.n_child[s] = nc;
    g.first_child[s] = nc > 0 ? blk[T] : 0;
    g.link[s] = (s == 0) ? 0 : rep[clink[T]];
    g.phi[s] = nphi[T];
    g.psi[s] = npsi[T];
    g.max_children = std::max(g.max_children, nc);
  }
  // root row: the root's arc on a token's class, else the root
  g.root_psi.assign(V + 1, 0.f);
  g.root_dst.assign(V + 1, 0);
  std::unordered_map<int32_t, int32_t> root_by_class;
  for (size_t j = 0; j < arcs[0].size(); ++j) root_by_class[arcs[0][j].first] = blk[0] + (int32_t)j;
  for (int32_t v = 0; v < V; ++v) {
    const auto it = root_by_class.find(class_map[v]);
    const int32_t d = it == root_by_class.end() ? 0 : it->second;
    g.root_dst[v] = d;
    g.root_psi[v] = g.psi[d];
  }
  return TB_OK;
}

}  // namespace

}  // namespace tbias

using namespace tbias;

extern "C" int tb_compile_variative(int32_t n_models, const int64_t* model_phrase_ptr,
                                    const int64_t* phrase_char_ptr, const int32_t* phrase_chars,
                                    const float* token_w, const float* end_bonus,
                                    const float* scale, const int64_t* token_char_ptr,
                                    const int32_t* token_chars, int32_t v_plus_blank,
                                    const int32_t* lower, int32_t n_chars, float tau,
                                    int32_t semantics, int32_t n_threads, tb_graphs** out) {
  if (!out) return fail(TB_EINVAL, "out is NULL");
  *out = nullptr;
  if (n_models < 1) return fail(TB_EINVAL, "n_models must be >= 1");
  if (!model_phrase_ptr || !phrase_char_ptr || !token_w || !end_bonus || !token_char_ptr ||
      !lower)
    return fail(TB_EINVAL, "NULL input array");
  if (v_plus_blank < 2) return fail(TB_EINVAL, "v_plus_blank must be >= 2");
  if (v_plus_blank > 32768) return fail(TB_ERANGE, "v_plus_blank must be <= 32768");
  if (n_chars < 1) return fail(TB_EINVAL, "n_chars must be >= 1");
  if (!std::isfinite(tau)) return fail(TB_EINVAL, "tau must be finite");
  if (semantics != TB_COMMIT && semantics != TB_PURE_POTENTIAL)
    return fail(TB_EINVAL, "unknown semantics");
  const int32_t V = v_plus_blank - 1;
  for (int32_t c = 0; c < n_chars; ++c)
    if (lower[c] < 0 || lower[c] >= n_chars)
      return fail(TB_ERANGE, "lower[" + std::to_string(c) + "] outside [0, n_chars)");
  if (token_char_ptr[0] != 0) return fail(TB_EINVAL, "token_char_ptr[0] != 0");
  for (int32_t v = 0; v < V; ++v)
    if (token_char_ptr[v + 1] <= token_char_ptr[v])
      return fail(token_char_ptr[v + 1] < token_char_ptr[v] ? TB_EINVAL : TB_ERANGE,
                  "token " + std::to_string(v) + " has no characters (or a decreasing CSR)");
  if (!token_chars) return fail(TB_EINVAL, "token_chars NULL");
  for (int64_t i = 0; i < token_char_ptr[V]; ++i)
    if (token_chars[i] < 0 || token_chars[i] >= n_chars)
      return fail(TB_ERANGE, "token character outside [0, n_chars)");
  if (model_phrase_ptr[0] != 0) return fail(TB_EINVAL, "model_phrase_ptr[0] != 0");
  for (int32_t m = 0; m < n_models; ++m)
    if (model_phrase_ptr[m + 1] < model_phrase_ptr[m])
      return fail(TB_EINVAL, "model_phrase_ptr not monotone");
  const int64_t n_phr = model_phrase_ptr[n_models];
  if (phrase_char_ptr[0] != 0) return fail(TB_EINVAL, "phrase_char_ptr[0] != 0");
  for (int64_t p = 0; p < n_phr; ++p)
    if (phrase_char_ptr[p + 1] < phrase_char_ptr[p])
      return fail(TB_EINVAL, "phrase_char_ptr not monotone");
  if (phrase_char_ptr[n_phr] > 0 && !phrase_chars) return fail(TB_EINVAL, "phrase_chars NULL");
  for (int64_t p = 0; p < n_phr; ++p) {
    if (phrase_char_ptr[p + 1] == phrase_char_ptr[p])
      return fail(TB_ERANGE, "empty phrase " + std::to_string(p));
    for (int64_t i = phrase_char_ptr[p]; i < phrase_char_ptr[p + 1]; ++i)
      if (phrase_chars[i] < 0 || phrase_chars[i] >= n_chars)
        return fail(TB_ERANGE, "phrase character outside [0, n_chars)");
  }

  // piece classes and the lowercased piece trie
  std::vector<int32_t> class_map(v_plus_blank, -1);
  PieceTrie pt;
  try {
    for (int32_t v = 0; v < V; ++v) {
      int32_t q = 0;
      for (int64_t i = token_char_ptr[v]; i < token_char_ptr[v + 1]; ++i) {
        const int32_t c = lower[token_chars[i]];
        int32_t r = pt.child(q, c);
        if (r < 0) {
          r = (int32_t)pt.next.size();
          pt.next.emplace_back();
          pt.cls.push_back(-1);
          pt.next[q][c] = r;
        }
        q = r;
      }
      if (pt.cls[q] < 0) pt.cls[q] = v;  // the smallest id with this string
      class_map[v] = pt.cls[q];
    }
  } catch (const std::bad_alloc&) {
    return fail(TB_ENOMEM, "host allocation failed");
  }

  std::vector<ModelGraph> graphs(n_models);
  std::vector<int> status(n_models, TB_OK);
  std::vector<std::string> errs(n_models);
  std::atomic<int32_t> next{0};
  int nt = n_threads > 0 ? n_threads : (int)std::thread::hardware_concurrency();
  nt = std::max(1, std::min(nt, n_models));
  auto work = [&]() {
    for (;;) {
      const int32_t m = next.fetch_add(1);
      if (m >= n_models) break;
      try {
        // lowercase, then sort and deduplicate the phrases
        std::vector<std::vector<int32_t>> ph;
        for (int64_t p = model_phrase_ptr[m]; p < model_phrase_ptr[m + 1]; ++p) {
          std::vector<int32_t> s;
          for (int64_t i = phrase_char_ptr[p]; i < phrase_char_ptr[p + 1]; ++i)
            s.push_back(lower[phrase_chars[i]]);
          ph.push_back(std::move(s));
        }
        std::sort(ph.begin(), ph.end());
        ph.erase(std::unique(ph.begin(), ph.end()), ph.end());
        const double a = scale ? (double)scale[m] : 1.0;
        status[m] = compile_variative_model(ph, pt, class_map.data(), V, (double)token_w[m],
                                            (double)end_bonus[m], a, (double)tau, semantics,
                                            &graphs[m]);
        if (status[m] != TB_OK) errs[m] = tb_last_error();
      } catch (const std::bad_alloc&) {
        status[m] = TB_ENOMEM;
        errs[m] = "host allocation failed while compiling";
      }
    }
  };
  if (nt == 1) {
    work();
  } else {
    std::vector<std::thread> pool;
    for (int i = 0; i < nt; ++i) pool.emplace_back(work);
    for (auto& t : pool) t.join();
  }
  for (int32_t m = 0; m < n_models; ++m)
    if (status[m] != TB_OK) return fail(status[m], "model " + std::to_string(m) + ": " + errs[m]);
  return assemble_image(graphs, class_map.data(), v_plus_blank, out);
}
