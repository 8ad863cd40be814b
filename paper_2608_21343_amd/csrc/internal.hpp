// Internal declarations shared by the host graph compiler and the C-ABI shim.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/tbias.h"

struct tb_graphs {
  tb_arena_layout layout;
  std::vector<unsigned char> image;  // exactly layout.total_bytes bytes
};

namespace tbias {

// thread-local error message
void set_error(const std::string& msg);
int fail(int code, const std::string& msg);

// per-model compile result (local ids, breadth-first numbering)
struct ModelGraph {
  int32_t n = 1;
  std::vector<int32_t> first_child, n_child, link, label;
  std::vector<float> phi, psi;
  std::vector<float> root_psi;    // V+1
  std::vector<int32_t> root_dst;  // V+1
  int32_t max_children = 0;
  int32_t max_depth = 0;
};

// Compile one model's phrase list (already validated token ids).
// Returns TB_OK or a negative code (message via set_error).
int compile_model(const int32_t* toks, const int64_t* tok_ptr, int64_t n_phrases,
                  const int32_t* class_map, int32_t V, double w, double bonus, double alpha,
                  int32_t semantics, ModelGraph* out);

inline int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

}  // namespace tbias
