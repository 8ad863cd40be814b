// Internal declarations shared by the host graph compiler and the C-ABI shim.
#pragma once

#include <cstdint>
#include <functional>
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
int assemble_image(const std::vector<const ModelGraph*>& graphs, const int32_t* class_map,
                   int32_t v_plus_blank, tb_graphs** out);

// The argument checks of tb_compile_graphs (same codes and messages).
int check_compile_args(int32_t n_models, const int64_t* model_phrase_ptr,
                       const int64_t* phrase_tok_ptr, const int32_t* phrase_tokens,
                       const float* token_w, const float* end_bonus, const int32_t* class_map,
                       int32_t v_plus_blank, int32_t semantics);

// Runs job(m) for every model m on up to n_threads host threads (<= 0:
// hardware concurrency); the first failing model's code, with its message.
int run_models(int32_t n_models, int32_t n_threads, const std::function<int(int32_t)>& job);

// The most tokens any state of the image overrides: the members of the
// classes of the children along its suffix chain, each class once (the
// image's links must end at the root).
int32_t image_max_override(const unsigned char* img, const tb_arena_layout& L);

inline int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

// Offsets (256-byte aligned) and total size of an arena image holding
// n_models model slots and n_states states; the maxima fields are left alone.
void plan_layout(int32_t n_models, int64_t n_states, int32_t v_plus_blank, tb_arena_layout* L);

// Class member CSR of a class map: members of class c are
// cls_tok[cls_ptr[c] .. cls_ptr[c+1]-1], ascending (cls_ptr has V+1 entries).
void class_tables(const int32_t* class_map, int32_t V, int32_t* cls_ptr, int32_t* cls_tok);

}  // namespace tbias
