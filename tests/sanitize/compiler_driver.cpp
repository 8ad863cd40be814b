// Host-side driver of the graph compilers, the image validator and the model
// caches, built with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_sanitize_cpu.py (no GPU code is involved: compiler.cpp,
// variative.cpp, cache.cpp and errors.cpp only).
//
// It compiles random phrase lists (empty lists, duplicates, nested and long
// phrases, case classes, several reading flags and thread counts), checks
// that every compiled image validates, corrupts images byte by byte and
// checks that validation rejects or accepts them without any memory error,
// and drives every documented argument error of tb_compile_graphs. The
// host-memory cache is driven with overlapping random lists under small
// budgets, every result compared with a fresh compile; saved files are
// loaded back and damaged (header fields, image bytes with and without a
// matching checksum) to check that loading refuses them cleanly.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <string>
#include <vector>

#include "../../include/tbias.h"

namespace {

int g_fail = 0;

void expect(bool ok, const char* what) {
  if (!ok) {
    std::fprintf(stderr, "FAIL: %s (%s)\n", what, tb_last_error());
    ++g_fail;
  }
}

struct Lists {
  std::vector<int64_t> mp{0}, tp{0};
  std::vector<int32_t> tok;
  void add_model(const std::vector<std::vector<int32_t>>& phrases) {
    for (const auto& p : phrases) {
      tok.insert(tok.end(), p.begin(), p.end());
      tp.push_back((int64_t)tok.size());
    }
    mp.push_back((int64_t)tp.size() - 1);
  }
  int32_t n_models() const { return (int32_t)mp.size() - 1; }
};

std::vector<int32_t> class_map(int32_t V, int32_t n_case) {
  std::vector<int32_t> cm(V + 1);
  for (int32_t v = 0; v < V; ++v) cm[v] = (v < 3 * n_case) ? v % n_case : v;
  cm[V] = -1;
  return cm;
}

tb_graphs* compile(const Lists& L, const std::vector<int32_t>& cm, int32_t sem, int32_t threads,
                   int* rc) {
  std::vector<float> w(L.n_models(), 1.0f), be(L.n_models(), 2.0f), sc(L.n_models(), 1.5f);
  tb_graphs* g = nullptr;
  *rc = tb_compile_graphs(L.n_models(), L.mp.data(), L.tp.data(),
                          L.tok.empty() ? nullptr : L.tok.data(), w.data(), be.data(),
                          (threads & 1) ? sc.data() : nullptr, cm.data(), (int32_t)cm.size(), sem,
                          threads, &g);
  return g;
}

void random_models(std::mt19937& rng) {
  std::uniform_int_distribution<int> nm(1, 6), np(0, 40), plen(1, 14);
  const int32_t V = 40 + (int32_t)(rng() % 300);
  const int32_t n_case = 1 + (int32_t)(rng() % (V / 3));
  std::uniform_int_distribution<int32_t> tokd(0, V - 1), small(0, 5);
  const auto cm = class_map(V, n_case);
  Lists L;
  const int M = nm(rng);
  for (int m = 0; m < M; ++m) {
    std::vector<std::vector<int32_t>> ph;
    const int n = (m == 0) ? 0 : np(rng);  // model 0: an empty list
    for (int i = 0; i < n; ++i) {
      std::vector<int32_t> p(plen(rng));
      const bool narrow = (rng() & 3) == 0;   // few symbols: deep shared prefixes
      for (auto& t : p) t = narrow ? small(rng) : tokd(rng);
      ph.push_back(p);
      if ((rng() & 7) == 0) ph.push_back(p);  // duplicates
      if ((rng() & 7) == 0 && p.size() > 1)   // nested prefixes
        ph.push_back(std::vector<int32_t>(p.begin(), p.begin() + p.size() / 2));
    }
    L.add_model(ph);
  }
  for (int32_t sem = 0; sem < 2; ++sem) {
    int rc = 0;
    tb_graphs* g = compile(L, cm, sem, 1 + (int32_t)(rng() % 4), &rc);
    expect(rc == TB_OK && g, "compile random models");
    if (!g) continue;
    tb_arena_layout lay;
    expect(tb_graphs_layout(g, &lay) == TB_OK, "layout");
    std::vector<unsigned char> img(lay.total_bytes);
    expect(tb_graphs_host_image(g, img.data(), lay.total_bytes) == TB_OK, "host image");
    expect(tb_graphs_host_image(g, img.data(), lay.total_bytes - 1) != TB_OK, "short buffer");
    expect(tb_validate_image(img.data(), &lay) == TB_OK, "validate compiled image");
    // corrupt single words: validation must never read out of bounds
    std::uniform_int_distribution<int64_t> pos(0, lay.total_bytes / 4 - 1);
    for (int k = 0; k < 64; ++k) {
      std::vector<unsigned char> bad = img;
      const int64_t i = pos(rng);
      const uint32_t vals[] = {0xffffffffu, 0x7fffffffu, 0x80000000u, 0u, (uint32_t)rng()};
      std::memcpy(bad.data() + 4 * i, &vals[rng() % 5], 4);
      const int r = tb_validate_image(bad.data(), &lay);
      expect(r == TB_OK || r == TB_ERANGE, "validate corrupted image returns a status");
    }
    tb_graphs_free(g);
  }
}

// Variative graphs: random piece vocabularies over a small alphabet (every
// character a piece, plus merged pieces, some of them cased), random phrase
// lists; the image must validate and survive single-word corruption.
void random_variative(std::mt19937& rng) {
  const int32_t n_low = 3 + (int32_t)(rng() % 6);  // lowercase letters; then their uppercase
  const int32_t n_chars = 2 * n_low;
  std::vector<int32_t> lower(n_chars);
  for (int32_t c = 0; c < n_chars; ++c) lower[c] = c % n_low;
  std::vector<std::vector<int32_t>> toks;
  for (int32_t c = 0; c < n_chars; ++c) toks.push_back({c});
  const int n_merged = (int)(rng() % 60);
  for (int i = 0; i < n_merged; ++i) {
    std::vector<int32_t> t(2 + rng() % 5);
    for (auto& c : t) c = (int32_t)(rng() % n_chars);
    toks.push_back(t);
  }
  std::vector<int64_t> tp{0};
  std::vector<int32_t> tc;
  for (const auto& t : toks) {
    tc.insert(tc.end(), t.begin(), t.end());
    tp.push_back((int64_t)tc.size());
  }
  const int32_t V1 = (int32_t)toks.size() + 1;
  Lists L;
  const int M = 1 + (int)(rng() % 4);
  for (int m = 0; m < M; ++m) {
    std::vector<std::vector<int32_t>> ph;
    const int n = (m == 0) ? 0 : (int)(rng() % 30);
    for (int i = 0; i < n; ++i) {
      std::vector<int32_t> p(1 + rng() % 12);
      for (auto& c : p) c = (int32_t)(rng() % ((rng() & 1) ? 2 : n_chars));
      ph.push_back(p);
      if ((rng() & 7) == 0) ph.push_back(p);
    }
    L.add_model(ph);
  }
  const float taus[] = {0.f, 0.5f, 1.f, 2.f};
  for (int32_t sem = 0; sem < 2; ++sem) {
    std::vector<float> w(L.n_models(), 1.0f), be(L.n_models(), 2.0f);
    tb_graphs* g = nullptr;
    const int rc = tb_compile_variative(L.n_models(), L.mp.data(), L.tp.data(),
                                        L.tok.empty() ? nullptr : L.tok.data(), w.data(), be.data(),
                                        nullptr, tp.data(), tc.data(), V1, lower.data(), n_chars,
                                        taus[rng() % 4], sem, 1 + (int32_t)(rng() % 3), &g);
    expect(rc == TB_OK && g, "compile random variative lists");
    if (!g) continue;
    tb_arena_layout lay;
    expect(tb_graphs_layout(g, &lay) == TB_OK, "variative layout");
    std::vector<unsigned char> img(lay.total_bytes);
    expect(tb_graphs_host_image(g, img.data(), lay.total_bytes) == TB_OK, "variative image");
    expect(tb_validate_image(img.data(), &lay) == TB_OK, "validate variative image");
    std::uniform_int_distribution<int64_t> pos(0, lay.total_bytes / 4 - 1);
    for (int k = 0; k < 64; ++k) {
      std::vector<unsigned char> bad = img;
      const uint32_t vals[] = {0xffffffffu, 0x7fffffffu, 0x80000000u, 0u, 1u, (uint32_t)rng()};
      std::memcpy(bad.data() + 4 * pos(rng), &vals[rng() % 6], 4);
      const int r = tb_validate_image(bad.data(), &lay);
      expect(r == TB_OK || r == TB_ERANGE, "validate corrupted variative image returns a status");
    }
    tb_graphs_free(g);
  }
  // a phrase character without a single-character piece
  {
    std::vector<int64_t> tp2{0, 2};
    std::vector<int32_t> tc2{0, 1};
    std::vector<int32_t> lw{0, 1};
    std::vector<int64_t> mp{0, 1}, pp{0, 2};
    std::vector<int32_t> pc{0, 1};
    std::vector<float> one(1, 1.f);
    tb_graphs* g = nullptr;
    expect(tb_compile_variative(1, mp.data(), pp.data(), pc.data(), one.data(), one.data(), nullptr,
                                tp2.data(), tc2.data(), 2, lw.data(), 2, 1.f, 0, 1, &g) ==
               TB_ERANGE, "missing character piece");
  }
}

std::vector<unsigned char> image_of(const tb_graphs* g, tb_arena_layout* lay) {
  tb_graphs_layout(g, lay);
  std::vector<unsigned char> img(lay->total_bytes);
  tb_graphs_host_image(g, img.data(), lay->total_bytes);
  return img;
}

// Overlapping random lists through one cache (budget from none to ample),
// every result equal to a fresh compile.
void random_cache(std::mt19937& rng) {
  const int32_t V = 40 + (int32_t)(rng() % 200);
  const auto cm = class_map(V, 1 + (int32_t)(rng() % (V / 3)));
  std::uniform_int_distribution<int32_t> tokd(0, V - 1);
  std::vector<std::vector<std::vector<int32_t>>> pool(8);
  for (auto& lst : pool) {
    const int n = (int)(rng() % 12);
    for (int i = 0; i < n; ++i) {
      std::vector<int32_t> p(1 + rng() % 6);
      for (auto& t : p) t = tokd(rng);
      lst.push_back(p);
    }
  }
  const int64_t caps[] = {0, 2000, 20000, 1 << 24};
  tb_graphs_cache* c = nullptr;
  expect(tb_graphs_cache_create(cm.data(), (int32_t)cm.size(), caps[rng() % 4], &c) == TB_OK,
         "cache create");
  if (!c) return;
  for (int round = 0; round < 6; ++round) {
    Lists L;
    const int M = 1 + (int)(rng() % 5);
    for (int m = 0; m < M; ++m) L.add_model(pool[rng() % pool.size()]);
    const int32_t sem = (int32_t)(rng() & 1), threads = 1 + (int32_t)(rng() % 4);
    std::vector<float> w(M, 1.0f), be(M, 2.0f), sc(M, 1.5f);
    const float* scp = (rng() & 1) ? sc.data() : nullptr;
    tb_graphs* a = nullptr;
    tb_graphs* b = nullptr;
    int32_t hits = -1;
    const int ra = tb_graphs_cache_compile(c, M, L.mp.data(), L.tp.data(),
                                           L.tok.empty() ? nullptr : L.tok.data(), w.data(),
                                           be.data(), scp, sem, threads, &hits, &a);
    const int rb = tb_compile_graphs(M, L.mp.data(), L.tp.data(),
                                     L.tok.empty() ? nullptr : L.tok.data(), w.data(), be.data(),
                                     scp, cm.data(), (int32_t)cm.size(), sem, threads, &b);
    expect(ra == TB_OK && rb == TB_OK && hits >= 0 && hits <= M, "cached and fresh compile");
    if (a && b) {
      tb_arena_layout la, lb;
      const auto ia = image_of(a, &la), ib = image_of(b, &lb);
      expect(std::memcmp(&la, &lb, sizeof la) == 0 && ia == ib, "cached compile equals fresh");
    }
    tb_graphs_free(a);
    tb_graphs_free(b);
  }
  int64_t st[5];
  expect(tb_graphs_cache_stats(c, st) == TB_OK && st[0] + st[1] > 0, "cache stats");
  expect(tb_graphs_cache_compile(nullptr, 1, nullptr, nullptr, nullptr, nullptr, nullptr,
                                 nullptr, 0, 1, nullptr, nullptr) == TB_EINVAL, "NULL cache");
  tb_graphs_cache_free(c);
}

uint64_t fnv1a64(const unsigned char* p, size_t n) {
  uint64_t h = 0xcbf29ce484222325ull;
  for (size_t i = 0; i < n; ++i) h = (h ^ p[i]) * 0x100000001b3ull;
  return h;
}

bool write_file(const std::string& path, const std::vector<unsigned char>& bytes) {
  FILE* f = std::fopen(path.c_str(), "wb");
  if (!f) return false;
  const bool ok = bytes.empty() || std::fwrite(bytes.data(), bytes.size(), 1, f) == 1;
  return std::fclose(f) == 0 && ok;
}

std::vector<unsigned char> read_file(const std::string& path) {
  std::vector<unsigned char> out;
  FILE* f = std::fopen(path.c_str(), "rb");
  if (!f) return out;
  unsigned char buf[65536];
  size_t n;
  while ((n = std::fread(buf, 1, sizeof buf, f)) > 0) out.insert(out.end(), buf, buf + n);
  std::fclose(f);
  return out;
}

// Save, load back, then load damaged copies: every load returns a status
// and never touches memory out of bounds.
void files(std::mt19937& rng, const std::string& dir) {
  const int32_t V = 60;
  const auto cm = class_map(V, 12);
  Lists L;
  L.add_model({{1, 2, 3}, {4, 5}, {1, 2, 9}});
  L.add_model({});
  L.add_model({{7}, {7, 8, 9, 10}, {8, 9}});
  int rc = 0;
  tb_graphs* g = compile(L, cm, 0, 2, &rc);
  expect(rc == TB_OK && g, "compile for files");
  if (!g) return;
  const std::string path = dir + "/driver.tbg";
  expect(tb_graphs_save(g, path.c_str()) == TB_OK, "save");
  tb_graphs* back = nullptr;
  expect(tb_graphs_load(path.c_str(), &back) == TB_OK && back, "load");
  tb_arena_layout lg, lb;
  if (back) {
    const auto ig = image_of(g, &lg), ib = image_of(back, &lb);
    expect(std::memcmp(&lg, &lb, sizeof lg) == 0 && ig == ib, "load equals save");
    tb_graphs_free(back);
  }
  const auto raw = read_file(path);
  const size_t head = 32 + sizeof(tb_arena_layout);
  expect(raw.size() == head + (size_t)lg.total_bytes, "file size");
  const std::string bad = dir + "/bad.tbg";
  std::uniform_int_distribution<size_t> anyb(0, raw.size() - 1), headb(0, head - 1);
  for (int k = 0; k < 200; ++k) {
    auto d = raw;
    const int kind = k % 4;
    if (kind == 0) {  // a header byte
      d[headb(rng)] ^= (unsigned char)(1 + rng() % 255);
    } else if (kind == 1) {  // an image byte, checksum left stale
      d[anyb(rng)] ^= (unsigned char)(1 + rng() % 255);
    } else if (kind == 2) {  // an image word, checksum updated: validation decides
      const size_t i = head + 4 * (rng() % ((raw.size() - head) / 4));
      const uint32_t vals[] = {0xffffffffu, 0x7fffffffu, 0x80000000u, 0u, (uint32_t)rng()};
      std::memcpy(d.data() + i, &vals[rng() % 5], 4);
      const uint64_t h = fnv1a64(d.data() + head, d.size() - head);
      std::memcpy(d.data() + 24, &h, 8);
    } else {  // truncated or extended
      d.resize((rng() & 1) ? rng() % raw.size() : raw.size() + 1 + rng() % 64);
    }
    expect(write_file(bad, d), "write damaged file");
    tb_graphs* x = nullptr;
    const int r = tb_graphs_load(bad.c_str(), &x);
    expect(r == TB_OK || r == TB_ERANGE || r == TB_EIO || r == TB_ENOMEM,
           "damaged file gives a status");
    expect((r == TB_OK) == (x != nullptr), "graphs only on success");
    tb_graphs_free(x);
  }
  tb_graphs* x = nullptr;
  expect(tb_graphs_load((dir + "/missing.tbg").c_str(), &x) == TB_EIO && !x, "missing file");
  expect(tb_graphs_save(g, (dir + "/no/such/dir.tbg").c_str()) == TB_EIO, "unwritable path");
  expect(tb_graphs_save(nullptr, path.c_str()) == TB_EINVAL, "NULL graphs");
  expect(tb_graphs_load(nullptr, &x) == TB_EINVAL, "NULL path");
  std::remove(path.c_str());
  std::remove(bad.c_str());
  tb_graphs_free(g);
}

void argument_errors() {
  const int32_t V = 50;
  const auto cm = class_map(V, 10);
  Lists L;
  L.add_model({{1, 2, 3}, {4}});
  int rc = 0;
  tb_graphs* g = compile(L, cm, 0, 1, &rc);
  expect(rc == TB_OK, "valid compile");
  tb_graphs_free(g);

  std::vector<float> one(1, 1.0f);
  tb_graphs* out = nullptr;
  auto call = [&](int32_t n, const int64_t* mp, const int64_t* tp, const int32_t* tk,
                  const int32_t* c, int32_t v1, int32_t sem, tb_graphs** o) {
    return tb_compile_graphs(n, mp, tp, tk, one.data(), one.data(), nullptr, c, v1, sem, 1, o);
  };
  expect(call(1, L.mp.data(), L.tp.data(), L.tok.data(), cm.data(), V + 1, 0, nullptr) ==
             TB_EINVAL, "NULL out");
  expect(call(0, L.mp.data(), L.tp.data(), L.tok.data(), cm.data(), V + 1, 0, &out) ==
             TB_EINVAL, "no models");
  expect(call(1, nullptr, L.tp.data(), L.tok.data(), cm.data(), V + 1, 0, &out) == TB_EINVAL,
         "NULL model_phrase_ptr");
  expect(call(1, L.mp.data(), L.tp.data(), L.tok.data(), cm.data(), 1, 0, &out) == TB_EINVAL,
         "v_plus_blank < 2");
  expect(call(1, L.mp.data(), L.tp.data(), L.tok.data(), cm.data(), V + 1, 7, &out) ==
             TB_EINVAL, "unknown reading");
  std::vector<int64_t> dec_tp = {0, 3, 2};  // a decreasing CSR
  expect(call(1, L.mp.data(), dec_tp.data(), L.tok.data(), cm.data(), V + 1, 0, &out) ==
             TB_EINVAL, "non-monotone phrase_tok_ptr");
  std::vector<int32_t> tk = {1, 2, 3, V};  // token == V (the blank)
  std::vector<int64_t> tp = {0, 3, 4}, mp = {0, 2};
  expect(call(1, mp.data(), tp.data(), tk.data(), cm.data(), V + 1, 0, &out) == TB_ERANGE,
         "blank in a phrase");
  tk[3] = -1;
  expect(call(1, mp.data(), tp.data(), tk.data(), cm.data(), V + 1, 0, &out) == TB_ERANGE,
         "negative token");
  std::vector<int64_t> tp_empty = {0, 3, 3};
  tk[3] = 4;
  expect(call(1, mp.data(), tp_empty.data(), tk.data(), cm.data(), V + 1, 0, &out) ==
             TB_ERANGE, "empty phrase");
  auto cm2 = cm;
  cm2[4] = -1;  // a non-blank token without a class cannot be in a phrase
  expect(call(1, mp.data(), tp.data(), tk.data(), cm2.data(), V + 1, 0, &out) == TB_ERANGE,
         "classless token");
  cm2 = cm;
  cm2[7] = V + 3;  // class id outside [0, V)
  expect(call(1, mp.data(), tp.data(), tk.data(), cm2.data(), V + 1, 0, &out) == TB_ERANGE,
         "class out of range");
}

}  // namespace

int main(int argc, char** argv) {
  std::mt19937 rng(12345);
  for (int i = 0; i < 60; ++i) random_models(rng);
  for (int i = 0; i < 60; ++i) random_variative(rng);
  for (int i = 0; i < 30; ++i) random_cache(rng);
  files(rng, argc > 1 ? argv[1] : ".");
  argument_errors();
  if (g_fail) {
    std::fprintf(stderr, "%d failures\n", g_fail);
    return 1;
  }
  std::printf("sanitized compiler driver: ok\n");
  return 0;
}
