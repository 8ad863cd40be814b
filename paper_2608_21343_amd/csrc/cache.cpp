// Host-side caches of compiled models (Sec. II-B, lifecycle paragraph): the
// paper keeps precompiled boosting models on disk, compiled models in CPU
// memory to be copied into the merged GPU model on demand, and models
// registered with the decoder before a session. The last level is the
// registry (registry.hip); this file holds the other two:
//
//  * tb_graphs_cache: compiled models of one class map in host memory, one
//    entry per model (its one-model arena image), keyed by everything that
//    determines its compile result (phrase list, token weight, end bonus,
//    scale, reading) and compared exactly; least recently used entries are
//    dropped beyond a byte budget. tb_graphs_cache_compile concatenates the
//    one-model images of a call's models (cached or just compiled), which
//    gives exactly the image tb_compile_graphs assembles for them.
//  * tb_graphs_save / tb_graphs_load: an arena image in a file, with a header
//    that the loader checks against the layout the image's counts imply, a
//    checksum, and the full image validation.

#include <algorithm>
#include <cstddef>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <list>
#include <memory>
#include <mutex>
#include <new>
#include <string>
#include <string_view>
#include <thread>
#include <unordered_map>

#include "internal.hpp"

using tbias::fail;
using tbias::ModelGraph;

struct tb_graphs_cache {
  struct Entry {
    std::string key;
    std::shared_ptr<const tb_graphs> graph;  // the model's one-model image
    int64_t bytes;
  };
  int32_t v_plus_blank = 0;
  std::vector<int32_t> class_map;
  int64_t capacity = 0;
  std::mutex mu;
  std::list<Entry> lru;  // most recently used first
  std::unordered_map<std::string_view, std::list<Entry>::iterator> index;  // views of Entry::key
  int64_t bytes = 0, hits = 0, misses = 0, dropped = 0;
};

namespace {

// Everything besides the class map that decides a model's compile result.
std::string model_key(const int32_t* toks, const int64_t* tok_ptr, int64_t n_phrases, float w,
                      float bonus, float alpha, int32_t semantics) {
  std::string k;
  auto put = [&](const void* p, size_t n) { k.append(static_cast<const char*>(p), n); };
  put(&semantics, sizeof semantics);
  put(&w, sizeof w);
  put(&bonus, sizeof bonus);
  put(&alpha, sizeof alpha);
  put(&n_phrases, sizeof n_phrases);
  for (int64_t p = 0; p < n_phrases; ++p) {
    const int64_t len = tok_ptr[p + 1] - tok_ptr[p];
    put(&len, sizeof len);
    if (len > 0) put(toks + tok_ptr[p], 4 * (size_t)len);
  }
  return k;
}

// Adds (key, g) unless the key is present; drops least recently used entries
// beyond the budget. Caller holds c.mu.
void insert_locked(tb_graphs_cache& c, std::string&& key, std::shared_ptr<const tb_graphs> g) {
  if (c.index.count(std::string_view(key))) return;
  const int64_t b = (int64_t)g->image.size() + (int64_t)key.size() + 128;
  if (b > c.capacity) return;
  c.lru.push_front(tb_graphs_cache::Entry{std::move(key), std::move(g), b});
  auto it = c.lru.begin();
  c.index.emplace(std::string_view(it->key), it);
  c.bytes += b;
  while (c.bytes > c.capacity && !c.lru.empty()) {
    auto last = std::prev(c.lru.end());
    c.bytes -= last->bytes;
    c.index.erase(std::string_view(last->key));
    c.lru.erase(last);
    ++c.dropped;
  }
}

// The image of models[0..], each a one-model image of the same class map and
// vocabulary: per-state arrays appended, per-model rows and value tables in
// model order, the class tables of the first, the maxima over all. Equals
// assemble_image of the models' compile results.
int concat_images(const std::vector<const tb_graphs*>& models, tb_graphs** out) {
  const int32_t n_models = (int32_t)models.size();
  const tb_arena_layout& F = models[0]->layout;
  const int32_t V1 = F.v_plus_blank;
  auto* g = new (std::nothrow) tb_graphs();
  if (!g) return fail(TB_ENOMEM, "host allocation failed");
  std::unique_ptr<tb_graphs> own(g);
  tb_arena_layout& L = g->layout;
  std::memset(&L, 0, sizeof L);
  int64_t N = 0;
  for (const tb_graphs* m : models) {
    N += m->layout.n_states;
    L.max_children = std::max(L.max_children, m->layout.max_children);
    L.max_depth = std::max(L.max_depth, m->layout.max_depth);
    L.max_override = std::max(L.max_override, m->layout.max_override);
  }
  if (N > INT32_MAX) return fail(TB_ERANGE, "more than 2^31 states in total");
  tbias::plan_layout(n_models, N, V1, &L);
  try {
    g->image.assign((size_t)L.total_bytes, 0);
  } catch (const std::bad_alloc&) {
    return fail(TB_ENOMEM, "host allocation of the arena image failed");
  }
  unsigned char* img = g->image.data();
  const int64_t state_arrays[][2] = {  // offset member, bytes per state
      {offsetof(tb_arena_layout, off_first_child), 4}, {offsetof(tb_arena_layout, off_n_child), 4},
      {offsetof(tb_arena_layout, off_link), 4},        {offsetof(tb_arena_layout, off_label), 4},
      {offsetof(tb_arena_layout, off_phi), 4},         {offsetof(tb_arena_layout, off_psi), 4},
      {offsetof(tb_arena_layout, off_arc_mem), 8},     {offsetof(tb_arena_layout, off_state_rec), 12}};
  auto off_of = [](const tb_arena_layout& l, int64_t member) {
    return *reinterpret_cast<const int64_t*>(reinterpret_cast<const char*>(&l) + member);
  };
  int64_t s0 = 0;
  for (int32_t i = 0; i < n_models; ++i) {
    const tb_arena_layout& M = models[i]->layout;
    const unsigned char* src = models[i]->image.data();
    const int64_t n = M.n_states;
    reinterpret_cast<int32_t*>(img + L.off_model_off)[i] = (int32_t)s0;
    reinterpret_cast<int32_t*>(img + L.off_model_n)[i] = (int32_t)n;
    for (const auto& a : state_arrays)
      std::memcpy(img + off_of(L, a[0]) + a[1] * s0, src + off_of(M, a[0]), (size_t)(a[1] * n));
    std::memcpy(img + L.off_root_psi + 4 * (int64_t)i * V1, src + M.off_root_psi, 4 * (size_t)V1);
    std::memcpy(img + L.off_root_dst + 4 * (int64_t)i * V1, src + M.off_root_dst, 4 * (size_t)V1);
    std::memcpy(img + L.off_value_tab + 4 * 512 * (int64_t)i, src + M.off_value_tab, 4 * 512);
    s0 += n;
  }
  const unsigned char* f = models[0]->image.data();
  std::memcpy(img + L.off_class_map, f + F.off_class_map, 4 * (size_t)V1);
  std::memcpy(img + L.off_cls_ptr, f + F.off_cls_ptr, 4 * (size_t)V1);
  std::memcpy(img + L.off_cls_tok, f + F.off_cls_tok, 4 * (size_t)(V1 - 1));
  *out = own.release();
  return TB_OK;
}

}  // namespace

extern "C" int tb_graphs_cache_create(const int32_t* class_map, int32_t v_plus_blank,
                                      int64_t capacity_bytes, tb_graphs_cache** out) {
  if (!out) return fail(TB_EINVAL, "out is NULL");
  *out = nullptr;
  if (!class_map) return fail(TB_EINVAL, "class_map is NULL");
  if (capacity_bytes < 0) return fail(TB_EINVAL, "capacity_bytes must be >= 0");
  if (v_plus_blank < 2) return fail(TB_EINVAL, "v_plus_blank must be >= 2");
  if (v_plus_blank > 32768) return fail(TB_ERANGE, "v_plus_blank must be <= 32768");
  const int32_t V = v_plus_blank - 1;
  if (class_map[V] != -1) return fail(TB_ERANGE, "class_map[blank] must be -1");
  for (int32_t v = 0; v < V; ++v)
    if (class_map[v] < -1 || class_map[v] >= V)
      return fail(TB_ERANGE, "class_map[" + std::to_string(v) + "] outside [-1, V)");
  auto* c = new (std::nothrow) tb_graphs_cache();
  if (!c) return fail(TB_ENOMEM, "host allocation failed");
  try {
    c->class_map.assign(class_map, class_map + v_plus_blank);
  } catch (const std::bad_alloc&) {
    delete c;
    return fail(TB_ENOMEM, "host allocation failed");
  }
  c->v_plus_blank = v_plus_blank;
  c->capacity = capacity_bytes;
  *out = c;
  return TB_OK;
}

extern "C" int tb_graphs_cache_compile(tb_graphs_cache* c, int32_t n_models,
                                       const int64_t* model_phrase_ptr,
                                       const int64_t* phrase_tok_ptr,
                                       const int32_t* phrase_tokens, const float* token_w,
                                       const float* end_bonus, const float* scale,
                                       int32_t semantics, int32_t n_threads, int32_t* hits,
                                       tb_graphs** out) {
  if (!out) return fail(TB_EINVAL, "out is NULL");
  *out = nullptr;
  if (!c) return fail(TB_EINVAL, "cache is NULL");
  const int32_t* cm = c->class_map.data();
  const int32_t V1 = c->v_plus_blank, V = V1 - 1;
  const int st = tbias::check_compile_args(n_models, model_phrase_ptr, phrase_tok_ptr,
                                           phrase_tokens, token_w, end_bonus, cm, V1, semantics);
  if (st != TB_OK) return st;
  std::vector<std::shared_ptr<const tb_graphs>> got(n_models);
  std::vector<uint8_t> hit(n_models, 0);
  const int rc = tbias::run_models(n_models, n_threads, [&](int32_t m) -> int {
    const int64_t p0 = model_phrase_ptr[m], p1 = model_phrase_ptr[m + 1];
    const float alpha = scale ? scale[m] : 1.0f;
    std::string key = model_key(phrase_tokens, phrase_tok_ptr + p0, p1 - p0, token_w[m],
                                end_bonus[m], alpha, semantics);
    {
      std::lock_guard<std::mutex> lock(c->mu);
      auto it = c->index.find(std::string_view(key));
      if (it != c->index.end()) {
        c->lru.splice(c->lru.begin(), c->lru, it->second);
        got[m] = it->second->graph;
        ++c->hits;
        hit[m] = 1;
        return TB_OK;
      }
      ++c->misses;
    }
    std::vector<ModelGraph> mg(1);
    int r = tbias::compile_model(phrase_tokens, phrase_tok_ptr + p0, p1 - p0, cm, V,
                                 (double)token_w[m], (double)end_bonus[m], (double)alpha,
                                 semantics, &mg[0]);
    if (r != TB_OK) return r;
    tb_graphs* one = nullptr;
    r = tbias::assemble_image(mg, cm, V1, &one);
    if (r != TB_OK) return r;
    std::shared_ptr<const tb_graphs> g(one, [](const tb_graphs* p) { delete p; });
    got[m] = g;
    std::lock_guard<std::mutex> lock(c->mu);
    insert_locked(*c, std::move(key), std::move(g));
    return TB_OK;
  });
  if (rc != TB_OK) return rc;
  if (hits) {
    int32_t h = 0;
    for (uint8_t x : hit) h += x;
    *hits = h;
  }
  std::vector<const tb_graphs*> ptrs(n_models);
  for (int32_t m = 0; m < n_models; ++m) ptrs[m] = got[m].get();
  return concat_images(ptrs, out);
}

extern "C" int tb_graphs_cache_stats(tb_graphs_cache* c, int64_t* stats) {
  if (!c || !stats) return fail(TB_EINVAL, "NULL argument");
  std::lock_guard<std::mutex> lock(c->mu);
  stats[0] = c->hits;
  stats[1] = c->misses;
  stats[2] = (int64_t)c->lru.size();
  stats[3] = c->bytes;
  stats[4] = c->dropped;
  return TB_OK;
}

extern "C" void tb_graphs_cache_free(tb_graphs_cache* c) { delete c; }

// ---- files

namespace {

constexpr char kTag[8] = {'T', 'B', 'G', 'R', 'A', 'P', 'H', 'S'};
constexpr uint32_t kVersion = 1;

struct FileHead {
  char tag[8];
  uint32_t version;
  uint32_t layout_bytes;  // sizeof(tb_arena_layout)
  uint64_t image_bytes;
  uint64_t checksum;  // FNV-1a (64-bit) of the image
  tb_arena_layout layout;
};

// FNV-1a, 64-bit (Fowler, Noll and Vo): xor each byte in, then multiply by
// the FNV prime.
uint64_t fnv1a64(const unsigned char* p, size_t n) {
  uint64_t h = 0xcbf29ce484222325ull;
  for (size_t i = 0; i < n; ++i) {
    h ^= p[i];
    h *= 0x100000001b3ull;
  }
  return h;
}

bool same_offsets(const tb_arena_layout& a, const tb_arena_layout& b) {
  return a.total_bytes == b.total_bytes && a.off_model_off == b.off_model_off &&
         a.off_model_n == b.off_model_n && a.off_first_child == b.off_first_child &&
         a.off_n_child == b.off_n_child && a.off_link == b.off_link &&
         a.off_label == b.off_label && a.off_phi == b.off_phi && a.off_psi == b.off_psi &&
         a.off_root_psi == b.off_root_psi && a.off_root_dst == b.off_root_dst &&
         a.off_class_map == b.off_class_map && a.off_cls_ptr == b.off_cls_ptr &&
         a.off_cls_tok == b.off_cls_tok && a.off_arc_mem == b.off_arc_mem &&
         a.off_value_tab == b.off_value_tab && a.off_state_rec == b.off_state_rec;
}

struct File {
  FILE* f = nullptr;
  ~File() {
    if (f) std::fclose(f);
  }
};

}  // namespace

extern "C" int tb_graphs_save(const tb_graphs* g, const char* path) {
  if (!g || !path) return fail(TB_EINVAL, "NULL argument");
  if ((int64_t)g->image.size() != g->layout.total_bytes)
    return fail(TB_EINVAL, "graphs image size differs from its layout");
  FileHead h;
  std::memset(&h, 0, sizeof h);
  std::memcpy(h.tag, kTag, sizeof kTag);
  h.version = kVersion;
  h.layout_bytes = (uint32_t)sizeof(tb_arena_layout);
  h.image_bytes = (uint64_t)g->image.size();
  h.checksum = fnv1a64(g->image.data(), g->image.size());
  h.layout = g->layout;
  const std::string tmp = std::string(path) + ".tmp" +
                          std::to_string(std::hash<std::thread::id>{}(std::this_thread::get_id()));
  bool ok;
  {
    File f;
    f.f = std::fopen(tmp.c_str(), "wb");
    if (!f.f) return fail(TB_EIO, "cannot open " + tmp + " for writing");
    ok = std::fwrite(&h, sizeof h, 1, f.f) == 1 &&
         (g->image.empty() ||
          std::fwrite(g->image.data(), g->image.size(), 1, f.f) == 1) &&
         std::fflush(f.f) == 0;
    const int cl = std::fclose(f.f);
    f.f = nullptr;
    ok = ok && cl == 0;
  }
  if (!ok || std::rename(tmp.c_str(), path) != 0) {
    std::remove(tmp.c_str());
    return fail(TB_EIO, std::string("cannot write ") + path);
  }
  return TB_OK;
}

extern "C" int tb_graphs_load(const char* path, tb_graphs** out) {
  if (!out) return fail(TB_EINVAL, "out is NULL");
  *out = nullptr;
  if (!path) return fail(TB_EINVAL, "path is NULL");
  File f;
  f.f = std::fopen(path, "rb");
  if (!f.f) return fail(TB_EIO, std::string("cannot open ") + path);
  if (std::fseek(f.f, 0, SEEK_END) != 0) return fail(TB_EIO, std::string("cannot read ") + path);
  const long size = std::ftell(f.f);
  if (size < 0 || std::fseek(f.f, 0, SEEK_SET) != 0)
    return fail(TB_EIO, std::string("cannot read ") + path);
  FileHead h;
  if ((uint64_t)size < sizeof h || std::fread(&h, sizeof h, 1, f.f) != 1)
    return fail(TB_ERANGE, std::string(path) + " is too short for a graphs file");
  if (std::memcmp(h.tag, kTag, sizeof kTag) != 0)
    return fail(TB_ERANGE, std::string(path) + " is not a graphs file");
  if (h.version != kVersion || h.layout_bytes != sizeof(tb_arena_layout))
    return fail(TB_ERANGE, std::string(path) + ": unsupported graphs file version");
  const tb_arena_layout& L = h.layout;
  if (L.n_models < 1 || L.v_plus_blank < 2 || L.v_plus_blank > 32768 ||
      L.n_states < L.n_models || L.n_states > INT32_MAX || L.max_children < 0 ||
      L.max_depth < 0 || L.max_override < 0)
    return fail(TB_ERANGE, std::string(path) + ": bad layout counts");
  tb_arena_layout want;
  std::memset(&want, 0, sizeof want);
  tbias::plan_layout(L.n_models, L.n_states, L.v_plus_blank, &want);
  if (!same_offsets(L, want) || h.image_bytes != (uint64_t)L.total_bytes ||
      (uint64_t)size != sizeof h + h.image_bytes)
    return fail(TB_ERANGE, std::string(path) + ": layout and size disagree");
  auto* g = new (std::nothrow) tb_graphs();
  if (!g) return fail(TB_ENOMEM, "host allocation failed");
  std::unique_ptr<tb_graphs> own(g);
  try {
    g->image.resize((size_t)h.image_bytes);
  } catch (const std::bad_alloc&) {
    return fail(TB_ENOMEM, "host allocation of the arena image failed");
  }
  if (h.image_bytes > 0 && std::fread(g->image.data(), (size_t)h.image_bytes, 1, f.f) != 1)
    return fail(TB_EIO, std::string("cannot read ") + path);
  if (fnv1a64(g->image.data(), g->image.size()) != h.checksum)
    return fail(TB_ERANGE, std::string(path) + ": checksum mismatch");
  g->layout = L;
  const int v = tb_validate_image(g->image.data(), &g->layout);
  if (v != TB_OK) return fail(v, std::string(path) + ": " + tb_last_error());
  const int32_t* nc = reinterpret_cast<const int32_t*>(g->image.data() + L.off_n_child);
  int32_t max_children = 0;
  for (int64_t x = 0; x < L.n_states; ++x) max_children = std::max(max_children, nc[x]);
  if (max_children != L.max_children ||
      tbias::image_max_override(g->image.data(), L) != L.max_override ||
      (int64_t)L.max_depth > L.n_states)
    return fail(TB_ERANGE, std::string(path) + ": layout maxima disagree with the image");
  *out = own.release();
  return TB_OK;
}
