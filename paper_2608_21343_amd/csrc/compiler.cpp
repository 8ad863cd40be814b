// Host graph compiler: per-stream phrase lists -> one merged arena image.
//
// TurboBias 2.0 compiles every context list into a weighted acceptor (arc
// labels and targets; per-state arc ranges, suffix-link targets and weights,
// final weights) and concatenates all active models into merged storage with
// per-model offsets (Sec. II-B). Case-insensitive matching (Sec. II-A) is
// obtained by labelling arcs with token case classes instead of tokens.
//
// This compiler emits that storage in a form shaped for the GPU step:
// * states are numbered breadth first with children in ascending class
//   order, so the children of a state are a contiguous id range and the arc
//   into state y is identified by y itself (its label is label[y]);
// * arc and suffix-link weights are kept as state potentials: stepping from
//   s into x scores psi[x] - phi[s] (Sec. II-A: an arc scores the difference
//   of potentials), following a suffix link from x to y changes the pending
//   score by phi[y] - phi[x];
// * every model gets a dense root row over tokens (root move target and psi),
//   which is the part of the step that does not depend on the stream's state.
//
// Potentials ("commit" reading; the paper leaves their values open):
//   l(x)   = depth of the deepest state on x's own root path that ends a phrase
//   phi(x) = alpha*w*(|x| - l(x))
//   E(x)   = alpha*(w*(|x| - l(parent x)) + bonus)  if x ends a phrase
//            alpha*bonus                            elif a proper suffix of x does
//            0                                      otherwise
//   psi(x) = phi(x) + E(x)
// "pure potential" reading: phi(x) = alpha*w*|x|, E(x) = alpha*bonus when x or
// a proper suffix of x ends a phrase. Both computed in double, stored float.

#include <algorithm>
#include <atomic>
#include <cstring>
#include <functional>
#include <system_error>
#include <thread>

#include "internal.hpp"

namespace tbias {

namespace {

struct Node {
  int32_t parent;
  int32_t label;
  int32_t first_kid = -1;  // index into kids of the build trie
  int32_t n_kids = 0;
  bool final = false;
};

// Binary search for the child of state s (new ids) labelled c; -1 if none.
inline int32_t child_of(const ModelGraph& g, int32_t s, int32_t c) {
  int32_t lo = g.first_child[s], hi = lo + g.n_child[s];
  while (lo < hi) {
    int32_t mid = (lo + hi) >> 1;
    int32_t l = g.label[mid];
    if (l == c) return mid;
    if (l < c) lo = mid + 1; else hi = mid;
  }
  return -1;
}

// Per-model value tables (distinct psi and phi values, ascending) and the
// packed state records of one model (see state_rec in tbias.h). fc, nc, lk,
// lb, phi, psi and out point at the model's first state.
void state_records(int32_t n, const int32_t* fc, const int32_t* nc, const int32_t* lk,
                   const int32_t* lb, const float* phi, const float* psi, const int32_t* cls_ptr,
                   float vtab[512], uint32_t* out) {
  std::vector<float> vp(psi, psi + n), vf(phi, phi + n);
  for (auto* v : {&vp, &vf}) {
    std::sort(v->begin(), v->end());
    v->erase(std::unique(v->begin(), v->end()), v->end());
  }
  for (int i = 0; i < 512; ++i) vtab[i] = 0.f;
  for (size_t i = 0; i < vp.size() && i < 256; ++i) vtab[i] = vp[i];
  for (size_t i = 0; i < vf.size() && i < 256; ++i) vtab[256 + i] = vf[i];
  for (int32_t x = 0; x < n; ++x) {
    const size_t ip = std::lower_bound(vp.begin(), vp.end(), psi[x]) - vp.begin();
    const size_t iq = std::lower_bound(vf.begin(), vf.end(), phi[x]) - vf.begin();
    const int32_t f = nc[x] > 0 ? fc[x] : 0;
    const int32_t lab = lb[x];
    const int32_t ms = lab >= 0 ? cls_ptr[lab] : 0;
    const int32_t mc = lab >= 0 ? cls_ptr[lab + 1] - cls_ptr[lab] : 0;
    const bool flag = f >= 65536 || nc[x] >= 255 || lk[x] >= 65536 || ms >= 65536 || mc > 255 ||
                      ip >= 256 || iq >= 256;
    if (flag) {
      out[3 * (int64_t)x] = 0u;
      out[3 * (int64_t)x + 1] = 0u;
      out[3 * (int64_t)x + 2] = 0x80000000u;
      continue;
    }
    out[3 * (int64_t)x] = (uint32_t)f | ((uint32_t)nc[x] << 16) | ((uint32_t)ip << 24);
    out[3 * (int64_t)x + 1] = (uint32_t)lk[x] | ((uint32_t)ms << 16);
    out[3 * (int64_t)x + 2] =
        (uint32_t)mc | ((uint32_t)iq << 8) | ((uint32_t)(lab >= 0 ? lab : 0) << 16);
  }
}

}  // namespace

int compile_model(const int32_t* toks, const int64_t* tok_ptr, int64_t n_phrases,
                  const int32_t* class_map, int32_t V, double w, double bonus, double alpha,
                  int32_t semantics, ModelGraph* out) {
  // 1. case-fold every phrase to its class string
  std::vector<int32_t> cls;
  std::vector<int64_t> cptr(n_phrases + 1, 0);
  cls.reserve(tok_ptr[n_phrases] - tok_ptr[0]);
  for (int64_t p = 0; p < n_phrases; ++p) {
    int64_t a = tok_ptr[p], b = tok_ptr[p + 1];
    if (b <= a) return fail(TB_ERANGE, "empty phrase " + std::to_string(p));
    for (int64_t i = a; i < b; ++i) {
      int32_t t = toks[i];
      if (t < 0 || t >= V)
        return fail(TB_ERANGE, "token " + std::to_string(t) + " outside [0, V)");
      int32_t c = class_map[t];
      if (c < 0) return fail(TB_ERANGE, "token " + std::to_string(t) + " has class -1");
      cls.push_back(c);
    }
    cptr[p + 1] = (int64_t)cls.size();
  }

  // 2. sort class strings lexicographically, drop duplicates
  std::vector<int64_t> order(n_phrases);
  for (int64_t i = 0; i < n_phrases; ++i) order[i] = i;
  auto less = [&](int64_t x, int64_t y) {
    return std::lexicographical_compare(cls.begin() + cptr[x], cls.begin() + cptr[x + 1],
                                        cls.begin() + cptr[y], cls.begin() + cptr[y + 1]);
  };
  std::sort(order.begin(), order.end(), less);

  // 3. build the trie in sorted order: the kids of every node arrive in
  //    ascending label order, stored as consecutive runs per node.
  std::vector<Node> nodes;
  nodes.reserve(cls.size() + 1);
  nodes.push_back(Node{-1, -1});
  std::vector<std::vector<int32_t>> kids(1);
  std::vector<int32_t> path{0};  // node at each depth of the previous string
  std::vector<int32_t> prev;
  for (int64_t oi = 0; oi < n_phrases; ++oi) {
    int64_t p = order[oi];
    const int32_t* s = cls.data() + cptr[p];
    int64_t L = cptr[p + 1] - cptr[p];
    size_t lcp = 0;
    while (lcp < prev.size() && lcp < (size_t)L && prev[lcp] == s[lcp]) ++lcp;
    path.resize(lcp + 1);
    for (int64_t i = (int64_t)lcp; i < L; ++i) {
      int32_t par = path.back();
      int32_t id = (int32_t)nodes.size();
      nodes.push_back(Node{par, s[i]});
      kids.emplace_back();
      kids[par].push_back(id);
      path.push_back(id);
    }
    nodes[path[L]].final = true;
    prev.assign(s, s + L);
  }

  // 4. breadth-first renumbering; children of each state become contiguous
  const int32_t n = (int32_t)nodes.size();
  ModelGraph& g = *out;
  g.n = n;
  g.first_child.assign(n, 0);
  g.n_child.assign(n, 0);
  g.link.assign(n, 0);
  g.label.assign(n, -1);
  g.phi.assign(n, 0.f);
  g.psi.assign(n, 0.f);
  std::vector<int32_t> newid(n), oldid(n), parent(n, -1), depth(n, 0);
  std::vector<char> fin(n, 0);
  oldid[0] = 0;
  newid[0] = 0;
  int32_t next = 1;
  for (int32_t q = 0; q < n; ++q) {  // oldid grows as the queue
    int32_t o = oldid[q];
    g.first_child[q] = next;
    g.n_child[q] = (int32_t)kids[o].size();
    g.max_children = std::max(g.max_children, g.n_child[q]);
    for (int32_t k : kids[o]) {
      newid[k] = next;
      oldid[next] = k;
      parent[next] = q;
      depth[next] = depth[q] + 1;
      g.label[next] = nodes[k].label;
      ++next;
    }
    fin[q] = nodes[o].final ? 1 : 0;
  }
  for (int32_t q = 0; q < n; ++q) g.max_depth = std::max(g.max_depth, depth[q]);
  // a state without children gets first_child = n_child = 0 for tidiness
  for (int32_t q = 0; q < n; ++q)
    if (g.n_child[q] == 0) g.first_child[q] = 0;

  // 5. suffix links in breadth-first order
  for (int32_t y = 1; y < n; ++y) {
    int32_t x = parent[y], c = g.label[y];
    if (x == 0) { g.link[y] = 0; continue; }
    int32_t f = g.link[x];
    for (;;) {
      int32_t h = child_of(g, f, c);
      if (h >= 0) { g.link[y] = h; break; }
      if (f == 0) { g.link[y] = 0; break; }
      f = g.link[f];
    }
  }

  // 6. potentials
  std::vector<int32_t> ell(n, 0);
  std::vector<char> suf_final(n, 0);  // a proper suffix ends a phrase
  for (int32_t y = 1; y < n; ++y) {
    ell[y] = fin[y] ? depth[y] : ell[parent[y]];
    int32_t l = g.link[y];
    suf_final[y] = (l != 0) && (fin[l] || suf_final[l]);
    double phi, E;
    if (semantics == TB_COMMIT) {
      phi = alpha * w * double(depth[y] - ell[y]);
      if (fin[y]) E = alpha * (w * double(depth[y] - ell[parent[y]]) + bonus);
      else if (suf_final[y]) E = alpha * bonus;
      else E = 0.0;
    } else {
      phi = alpha * w * double(depth[y]);
      E = (fin[y] || suf_final[y]) ? alpha * bonus : 0.0;
    }
    g.phi[y] = (float)phi;
    g.psi[y] = (float)(phi + E);
  }

  // 7. dense root row over tokens
  std::vector<int32_t> root_by_class(V, 0);
  for (int32_t j = 0; j < g.n_child[0]; ++j) {
    int32_t y = g.first_child[0] + j;
    root_by_class[g.label[y]] = y;
  }
  g.root_psi.assign(V + 1, 0.f);
  g.root_dst.assign(V + 1, 0);
  for (int32_t v = 0; v < V; ++v) {
    int32_t c = class_map[v];
    int32_t d = (c >= 0) ? root_by_class[c] : 0;
    g.root_dst[v] = d;
    g.root_psi[v] = g.psi[d];
  }
  return TB_OK;
}

void plan_layout(int32_t n_models, int64_t n_states, int32_t v_plus_blank, tb_arena_layout* L) {
  const int64_t M = n_models, N = n_states, R = (int64_t)n_models * v_plus_blank;
  const int32_t V = v_plus_blank - 1;
  L->n_models = n_models;
  L->v_plus_blank = v_plus_blank;
  L->n_states = n_states;
  int64_t off = 0;
  auto take = [&](int64_t bytes) { int64_t o = off; off = align256(off + bytes); return o; };
  L->off_model_off = take(4 * M);
  L->off_model_n = take(4 * M);
  L->off_first_child = take(4 * N);
  L->off_n_child = take(4 * N);
  L->off_link = take(4 * N);
  L->off_label = take(4 * N);
  L->off_phi = take(4 * N);
  L->off_psi = take(4 * N);
  L->off_root_psi = take(4 * R);
  L->off_root_dst = take(4 * R);
  L->off_class_map = take(4 * (int64_t)v_plus_blank);
  L->off_cls_ptr = take(4 * (int64_t)v_plus_blank);
  L->off_cls_tok = take(4 * (int64_t)V);
  L->off_arc_mem = take(8 * N);
  L->off_value_tab = take(4 * 512 * M);
  L->off_state_rec = take(12 * N);
  L->total_bytes = off;
}

void class_tables(const int32_t* class_map, int32_t V, int32_t* cp, int32_t* ct) {
  // members ascending because tokens are scanned in order
  std::vector<int32_t> cnt(V + 1, 0);
  for (int32_t v = 0; v < V; ++v)
    if (class_map[v] >= 0) cnt[class_map[v] + 1]++;
  cp[0] = 0;
  for (int32_t c = 0; c < V; ++c) cp[c + 1] = cp[c] + cnt[c + 1];
  std::vector<int32_t> fillp(cp, cp + V);
  for (int32_t v = 0; v < V; ++v)
    if (class_map[v] >= 0) ct[fillp[class_map[v]]++] = v;
}

}  // namespace tbias

using namespace tbias;

namespace tbias {

int check_compile_args(int32_t n_models, const int64_t* model_phrase_ptr,
                       const int64_t* phrase_tok_ptr, const int32_t* phrase_tokens,
                       const float* token_w, const float* end_bonus, const int32_t* class_map,
                       int32_t v_plus_blank, int32_t semantics) {
  if (n_models < 1) return fail(TB_EINVAL, "n_models must be >= 1");
  if (!model_phrase_ptr || !phrase_tok_ptr || !token_w || !end_bonus || !class_map)
    return fail(TB_EINVAL, "NULL input array");
  if (v_plus_blank < 2) return fail(TB_EINVAL, "v_plus_blank must be >= 2");
  if (v_plus_blank > 32768) return fail(TB_ERANGE, "v_plus_blank must be <= 32768");
  if (semantics != TB_COMMIT && semantics != TB_PURE_POTENTIAL)
    return fail(TB_EINVAL, "unknown semantics");
  const int32_t V = v_plus_blank - 1;
  if (class_map[V] != -1) return fail(TB_ERANGE, "class_map[blank] must be -1");
  for (int32_t v = 0; v < V; ++v)
    if (class_map[v] < -1 || class_map[v] >= V)
      return fail(TB_ERANGE, "class_map[" + std::to_string(v) + "] outside [-1, V)");
  if (model_phrase_ptr[0] != 0) return fail(TB_EINVAL, "model_phrase_ptr[0] != 0");
  for (int32_t m = 0; m < n_models; ++m)
    if (model_phrase_ptr[m + 1] < model_phrase_ptr[m])
      return fail(TB_EINVAL, "model_phrase_ptr not monotone");
  const int64_t n_phr = model_phrase_ptr[n_models];
  if (phrase_tok_ptr[0] != 0) return fail(TB_EINVAL, "phrase_tok_ptr[0] != 0");
  for (int64_t p = 0; p < n_phr; ++p)
    if (phrase_tok_ptr[p + 1] < phrase_tok_ptr[p])
      return fail(TB_EINVAL, "phrase_tok_ptr not monotone");
  if (phrase_tok_ptr[n_phr] > 0 && !phrase_tokens) return fail(TB_EINVAL, "phrase_tokens NULL");
  return TB_OK;
}

int run_models(int32_t n_models, int32_t n_threads, const std::function<int(int32_t)>& job) {
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
        status[m] = job(m);
      } catch (const std::bad_alloc&) {
        status[m] = fail(TB_ENOMEM, "host allocation failed while compiling");
      }
      if (status[m] != TB_OK) errs[m] = tb_last_error();
    }
  };
  try {
    if (nt == 1) {
      work();
    } else {
      std::vector<std::thread> pool;
      for (int i = 0; i < nt; ++i) pool.emplace_back(work);
      for (auto& t : pool) t.join();
    }
  } catch (const std::system_error&) {
    return fail(TB_ENOMEM, "could not start the compile threads");
  }
  for (int32_t m = 0; m < n_models; ++m)
    if (status[m] != TB_OK)
      return fail(status[m], "model " + std::to_string(m) + ": " + errs[m]);
  return TB_OK;
}

}  // namespace tbias

extern "C" int tb_compile_graphs(int32_t n_models, const int64_t* model_phrase_ptr,
                                 const int64_t* phrase_tok_ptr, const int32_t* phrase_tokens,
                                 const float* token_w, const float* end_bonus, const float* scale,
                                 const int32_t* class_map, int32_t v_plus_blank,
                                 int32_t semantics, int32_t n_threads, tb_graphs** out) {
  if (!out) return fail(TB_EINVAL, "out is NULL");
  *out = nullptr;
  const int st = check_compile_args(n_models, model_phrase_ptr, phrase_tok_ptr, phrase_tokens,
                                    token_w, end_bonus, class_map, v_plus_blank, semantics);
  if (st != TB_OK) return st;
  const int32_t V = v_plus_blank - 1;
  std::vector<ModelGraph> graphs(n_models);
  const int rc = run_models(n_models, n_threads, [&](int32_t m) -> int {
    const int64_t p0 = model_phrase_ptr[m], p1 = model_phrase_ptr[m + 1];
    const double a = scale ? (double)scale[m] : 1.0;
    return compile_model(phrase_tokens, phrase_tok_ptr + p0, p1 - p0, class_map, V,
                         (double)token_w[m], (double)end_bonus[m], a, semantics, &graphs[m]);
  });
  if (rc != TB_OK) return rc;
  return assemble_image(graphs, class_map, v_plus_blank, out);
}

namespace tbias {

int assemble_image(const std::vector<ModelGraph>& graphs, const int32_t* class_map,
                   int32_t v_plus_blank, tb_graphs** out) {
  std::vector<const ModelGraph*> ptrs(graphs.size());
  for (size_t m = 0; m < graphs.size(); ++m) ptrs[m] = &graphs[m];
  return assemble_image(ptrs, class_map, v_plus_blank, out);
}

int assemble_image(const std::vector<const ModelGraph*>& graphs, const int32_t* class_map,
                   int32_t v_plus_blank, tb_graphs** out) {
  const int32_t n_models = (int32_t)graphs.size();
  const int32_t V = v_plus_blank - 1;
  auto* g = new (std::nothrow) tb_graphs();
  if (!g) return fail(TB_ENOMEM, "host allocation failed");
  tb_arena_layout& L = g->layout;
  std::memset(&L, 0, sizeof(L));
  int64_t N = 0;
  for (const ModelGraph* mg : graphs) {
    N += mg->n;
    L.max_children = std::max(L.max_children, mg->max_children);
    L.max_depth = std::max(L.max_depth, mg->max_depth);
  }
  if (N > INT32_MAX) { delete g; return fail(TB_ERANGE, "more than 2^31 states in total"); }
  plan_layout(n_models, N, v_plus_blank, &L);
  const int64_t off = L.total_bytes;
  try {
    g->image.assign((size_t)off, 0);
  } catch (const std::bad_alloc&) {
    delete g;
    return fail(TB_ENOMEM, "host allocation of the arena image failed");
  }
  unsigned char* img = g->image.data();
  auto I32 = [&](int64_t o) { return reinterpret_cast<int32_t*>(img + o); };
  auto F32 = [&](int64_t o) { return reinterpret_cast<float*>(img + o); };
  int64_t s0 = 0;
  for (int32_t m = 0; m < n_models; ++m) {
    const ModelGraph& mg = *graphs[m];
    I32(L.off_model_off)[m] = (int32_t)s0;
    I32(L.off_model_n)[m] = mg.n;
    std::memcpy(I32(L.off_first_child) + s0, mg.first_child.data(), 4 * (size_t)mg.n);
    std::memcpy(I32(L.off_n_child) + s0, mg.n_child.data(), 4 * (size_t)mg.n);
    std::memcpy(I32(L.off_link) + s0, mg.link.data(), 4 * (size_t)mg.n);
    std::memcpy(I32(L.off_label) + s0, mg.label.data(), 4 * (size_t)mg.n);
    std::memcpy(F32(L.off_phi) + s0, mg.phi.data(), 4 * (size_t)mg.n);
    std::memcpy(F32(L.off_psi) + s0, mg.psi.data(), 4 * (size_t)mg.n);
    std::memcpy(F32(L.off_root_psi) + (int64_t)m * v_plus_blank, mg.root_psi.data(),
                4 * (size_t)v_plus_blank);
    std::memcpy(I32(L.off_root_dst) + (int64_t)m * v_plus_blank, mg.root_dst.data(),
                4 * (size_t)v_plus_blank);
    s0 += mg.n;
  }
  std::memcpy(I32(L.off_class_map), class_map, 4 * (size_t)v_plus_blank);
  // class members CSR
  int32_t* cp = I32(L.off_cls_ptr);
  int32_t* ct = I32(L.off_cls_tok);
  class_tables(class_map, V, cp, ct);
  L.max_override = image_max_override(img, L);
  // member tokens of the class on the arc into every state (see arc_mem in tbias.h)
  uint32_t* am = reinterpret_cast<uint32_t*>(img + L.off_arc_mem);
  for (int64_t y = 0; y < N; ++y) {
    const int32_t lab = I32(L.off_label)[y];
    if (lab < 0) {  // a root
      am[2 * y] = 0u;
      am[2 * y + 1] = 0u;
      continue;
    }
    const int32_t m0 = cp[lab], nm = cp[lab + 1] - cp[lab];
    const uint32_t t0 = (uint32_t)ct[m0];
    const uint32_t t1 = (uint32_t)ct[m0 + (nm > 1 ? 1 : 0)];
    const uint32_t t2 = (uint32_t)ct[m0 + (nm > 2 ? 2 : nm - 1)];
    am[2 * y] = t0 | (t1 << 16);
    am[2 * y + 1] = t2 | ((uint32_t)lab << 16) | (nm > 3 ? 0x80000000u : 0u);
  }
  // value tables and packed state records
  for (int32_t m = 0; m < n_models; ++m) {
    const int32_t so = I32(L.off_model_off)[m];
    state_records(graphs[m]->n, I32(L.off_first_child) + so, I32(L.off_n_child) + so,
                  I32(L.off_link) + so, I32(L.off_label) + so, F32(L.off_phi) + so,
                  F32(L.off_psi) + so, cp, F32(L.off_value_tab) + 512 * (int64_t)m,
                  reinterpret_cast<uint32_t*>(img + L.off_state_rec) + 3 * (int64_t)so);
  }
  *out = g;
  return TB_OK;
}

}  // namespace tbias

extern "C" int tb_graphs_layout(const tb_graphs* g, tb_arena_layout* out) {
  if (!g || !out) return fail(TB_EINVAL, "NULL argument");
  *out = g->layout;
  return TB_OK;
}

extern "C" int tb_graphs_host_image(const tb_graphs* g, void* dst, int64_t bytes) {
  if (!g || !dst) return fail(TB_EINVAL, "NULL argument");
  if (bytes < g->layout.total_bytes) return fail(TB_ENOMEM, "destination too small");
  std::memcpy(dst, g->image.data(), (size_t)g->layout.total_bytes);
  return TB_OK;
}

extern "C" void tb_graphs_free(tb_graphs* g) { delete g; }

namespace tbias {

int32_t image_max_override(const unsigned char* img, const tb_arena_layout& L) {
  // over all states, the member tokens of the classes of the children along
  // the state's suffix chain (root excluded), each class counted once
  auto I32 = [&](int64_t o) { return reinterpret_cast<const int32_t*>(img + o); };
  const int32_t V = L.v_plus_blank - 1;
  const int32_t* cp = I32(L.off_cls_ptr);
  std::vector<int64_t> seen(V, -1);
  int64_t gen = 0;
  int32_t best = 0;
  for (int32_t m = 0; m < L.n_models; ++m) {
    const int32_t so = I32(L.off_model_off)[m], n = I32(L.off_model_n)[m];
    const int32_t* fc = I32(L.off_first_child) + so;
    const int32_t* nc = I32(L.off_n_child) + so;
    const int32_t* lk = I32(L.off_link) + so;
    const int32_t* lb = I32(L.off_label) + so;
    for (int32_t x = 1; x < n; ++x, ++gen) {
      int32_t members = 0;
      for (int32_t c = x; c != 0; c = lk[c])
        for (int32_t j = 0; j < nc[c]; ++j) {
          const int32_t lab = lb[fc[c] + j];
          if (seen[lab] == gen) continue;
          seen[lab] = gen;
          members += cp[lab + 1] - cp[lab];
        }
      best = std::max(best, members);
    }
  }
  return best;
}

}  // namespace tbias

extern "C" int tb_validate_image(const void* host_image, const tb_arena_layout* Lp) {
  if (!host_image || !Lp) return fail(TB_EINVAL, "NULL argument");
  const tb_arena_layout& L = *Lp;
  const unsigned char* img = static_cast<const unsigned char*>(host_image);
  auto I32 = [&](int64_t o) { return reinterpret_cast<const int32_t*>(img + o); };
  const int32_t V1 = L.v_plus_blank, V = V1 - 1;
  if (L.n_models < 1 || V1 < 2 || L.n_states < L.n_models)
    return fail(TB_ERANGE, "bad layout header");
  const int32_t* cm = I32(L.off_class_map);
  if (cm[V] != -1) return fail(TB_ERANGE, "class_map[blank] != -1");
  for (int32_t v = 0; v < V; ++v)
    if (cm[v] < -1 || cm[v] >= V) return fail(TB_ERANGE, "class_map entry out of range");
  int64_t expect_off = 0;
  for (int32_t m = 0; m < L.n_models; ++m) {
    int32_t off = I32(L.off_model_off)[m], n = I32(L.off_model_n)[m];
    if (off != expect_off || n < 1 || off + (int64_t)n > L.n_states)
      return fail(TB_ERANGE, "model table inconsistent at model " + std::to_string(m));
    expect_off += n;
    const int32_t* fc = I32(L.off_first_child) + off;
    const int32_t* nc = I32(L.off_n_child) + off;
    const int32_t* lk = I32(L.off_link) + off;
    const int32_t* lb = I32(L.off_label) + off;
    if (lk[0] != 0 || lb[0] != -1) return fail(TB_ERANGE, "bad root record");
    for (int32_t s = 0; s < n; ++s) {
      if (s > 0 && (lk[s] < 0 || lk[s] >= n))
        return fail(TB_ERANGE, "suffix link of state " + std::to_string(s) + " out of range");
      if (s > 0 && (lb[s] < 0 || lb[s] >= V))
        return fail(TB_ERANGE, "label of state " + std::to_string(s) + " out of range");
      // children are non-root states; several states may share one child range
      // (the arcs into one node of a variative graph)
      if (nc[s] < 0 || (nc[s] > 0 && (fc[s] < 1 || (int64_t)fc[s] + nc[s] > n)))
        return fail(TB_ERANGE, "child range of state " + std::to_string(s) + " out of range");
      for (int32_t j = 1; j < nc[s]; ++j)
        if (lb[fc[s] + j] <= lb[fc[s] + j - 1])
          return fail(TB_ERANGE, "children labels not ascending");
    }
    // every suffix chain ends at the root: no cycle among the links
    {
      std::vector<uint8_t> col(n, 0);  // 0 unseen, 1 on the current chain, 2 ends at the root
      std::vector<int32_t> chain;
      col[0] = 2;
      for (int32_t s = 1; s < n; ++s) {
        int32_t x = s;
        chain.clear();
        while (col[x] == 0) {
          col[x] = 1;
          chain.push_back(x);
          x = lk[x];
        }
        if (col[x] == 1)
          return fail(TB_ERANGE, "suffix links of model " + std::to_string(m) + " form a cycle");
        for (int32_t y : chain) col[y] = 2;
      }
    }
    // root rows: the root move of a token is the root's child on its class,
    // else the root itself; its psi is that state's psi; the blank column is 0
    const int32_t* rd = I32(L.off_root_dst) + (int64_t)m * V1;
    const float* rp = reinterpret_cast<const float*>(img + L.off_root_psi) + (int64_t)m * V1;
    const float* ps = reinterpret_cast<const float*>(img + L.off_psi) + off;
    std::vector<int32_t> child_on(V, 0);
    for (int32_t j = 0; j < nc[0]; ++j) child_on[lb[fc[0] + j]] = fc[0] + j;
    for (int32_t v = 0; v < V; ++v) {
      const int32_t want = cm[v] >= 0 ? child_on[cm[v]] : 0;
      if (rd[v] != want || !(rp[v] == ps[want]))
        return fail(TB_ERANGE, "root row of model " + std::to_string(m) + " inconsistent at token " +
                                   std::to_string(v));
    }
    if (rd[V] != 0 || rp[V] != 0.f) return fail(TB_ERANGE, "root row blank column not zero");
  }
  if (expect_off != L.n_states) return fail(TB_ERANGE, "state count mismatch");
  const int32_t* cp = I32(L.off_cls_ptr);
  if (cp[0] != 0) return fail(TB_ERANGE, "cls_ptr[0] != 0");
  for (int32_t c = 0; c < V; ++c)
    if (cp[c + 1] < cp[c] || cp[c + 1] > V) return fail(TB_ERANGE, "cls_ptr not monotone");
  // class members: every token of class c listed once under c, ascending
  const int32_t* ct = I32(L.off_cls_tok);
  int32_t n_member = 0;
  for (int32_t v = 0; v < V; ++v) n_member += cm[v] >= 0;
  if (cp[V] != n_member) return fail(TB_ERANGE, "cls_ptr total differs from the classed tokens");
  for (int32_t c = 0; c < V; ++c)
    for (int32_t q = cp[c]; q < cp[c + 1]; ++q)
      if (ct[q] < 0 || ct[q] >= V || cm[ct[q]] != c || (q > cp[c] && ct[q] <= ct[q - 1]))
        return fail(TB_ERANGE, "class member list of class " + std::to_string(c) + " inconsistent");
  // arc member records agree with the labels and the class member lists
  const uint32_t* am = reinterpret_cast<const uint32_t*>(img + L.off_arc_mem);
  const int32_t* lab_all = I32(L.off_label);
  for (int64_t y = 0; y < L.n_states; ++y) {
    const int32_t lab = lab_all[y];
    if (lab < 0) {
      if (am[2 * y] != 0u || am[2 * y + 1] != 0u) return fail(TB_ERANGE, "root arc record not zero");
      continue;
    }
    const int32_t m0 = cp[lab], nm = cp[lab + 1] - cp[lab];
    if (nm < 1) return fail(TB_ERANGE, "arc label of a class without members");
    const uint32_t t0 = (uint32_t)ct[m0];
    const uint32_t t1 = (uint32_t)ct[m0 + (nm > 1 ? 1 : 0)];
    const uint32_t t2 = (uint32_t)ct[m0 + (nm > 2 ? 2 : nm - 1)];
    const uint32_t w1 = t2 | ((uint32_t)lab << 16) | (nm > 3 ? 0x80000000u : 0u);
    if (am[2 * y] != (t0 | (t1 << 16)) || am[2 * y + 1] != w1)
      return fail(TB_ERANGE, "arc member record of state " + std::to_string(y) + " inconsistent");
  }
  // value tables and state records equal the ones derived from the arrays above
  {
    std::vector<uint32_t> want;
    float vt[512];
    for (int32_t m = 0; m < L.n_models; ++m) {
      const int32_t so = I32(L.off_model_off)[m], n = I32(L.off_model_n)[m];
      want.assign(3 * (size_t)n, 0u);
      state_records(n, I32(L.off_first_child) + so, I32(L.off_n_child) + so,
                    I32(L.off_link) + so, lab_all + so,
                    reinterpret_cast<const float*>(img + L.off_phi) + so,
                    reinterpret_cast<const float*>(img + L.off_psi) + so, cp, vt, want.data());
      const float* vimg = reinterpret_cast<const float*>(img + L.off_value_tab) + 512 * (int64_t)m;
      if (std::memcmp(vt, vimg, sizeof(vt)) != 0)
        return fail(TB_ERANGE, "value table of model " + std::to_string(m) + " inconsistent");
      const uint32_t* sr = reinterpret_cast<const uint32_t*>(img + L.off_state_rec) + 3 * (int64_t)so;
      for (int32_t x = 0; x < n; ++x)
        if (std::memcmp(&want[3 * (size_t)x], sr + 3 * (int64_t)x, 12) != 0)
          return fail(TB_ERANGE, "state record of state " + std::to_string(x) + " of model " +
                                     std::to_string(m) + " inconsistent");
    }
  }
  return TB_OK;
}
