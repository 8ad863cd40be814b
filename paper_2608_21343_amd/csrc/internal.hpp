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

// Concatenate compiled models into one arena image (offsets, class tables,
// arc member records, value tables, packed state records); *out owns it.
int assemble_image(const std::vector<ModelGraph>& graphs, const int32_t* class_map,
                   int32_t v_plus_blank, tb_graphs** out);

inline int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

// Offsets (256-byte aligned) and total size of an arena image holding
// n_models model slots and n_states states; the maxima fields are left alone.
void plan_layout(int32_t n_models, int64_t n_states, int32_t v_plus_blank, tb_arena_layout* L);

// Class member CSR of a class map: members of class c are
// cls_tok[cls_ptr[c] .. cls_ptr[c+1]-1], ascending (cls_ptr has V+1 entries).
void class_tables(const int32_t* class_map, int32_t V, int32_t* cls_ptr, int32_t* cls_tok);

}  // namespace tbias
