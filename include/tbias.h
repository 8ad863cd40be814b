/*
 * tbias.h — C ABI of the MI355X boosted-decode library (libtbias.so).
 *
 * Per-stream phrase boosting fused into batched Transducer greedy and beam
 * decoding, after TurboBias 2.0 (Sec. II). Every stream carries a boosting
 * model id (Sec. II-B; -1 = no biasing) and a graph state; one decoding step
 * adds the boosting score of every vocabulary token to the stream's joint
 * logits, normalises (log-softmax), selects (argmax or top-K) and advances the
 * graph state, which is carried across streaming calls (Sec. II-C).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every function returns an int status: TB_OK (0) or a negative TB_E* code.
 *   tb_last_error() returns a thread-local message for the last failure.
 * - Argument checks are synchronous and happen before any launch: a call that
 *   returns an error has enqueued nothing.
 * - "device" pointers are HIP device memory owned by the caller (the library
 *   never allocates device memory); "host" pointers are ordinary host memory.
 *   Kernels run asynchronously on the given HIP stream (NULL = the default
 *   stream); outputs are valid once that stream has reached the call.
 * - The vocabulary has V non-blank tokens with ids 0..V-1 and the blank with
 *   id V (the last logit column); v_plus_blank = V + 1.
 * - Graph states are model-local breadth-first ids (root = 0); -1 means "no
 *   model". A carried state or model id that is out of range for the arena is
 *   never dereferenced: that stream is decoded without biasing and its output
 *   states are written as TB_STATE_INVALID (-2), or TB_STATE_TIMEOUT (-3) when
 *   the carried state was TB_STATE_TIMEOUT (see below).
 */
#ifndef TBIAS_H
#define TBIAS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  TB_OK = 0,
  TB_EINVAL = -1, /* bad argument (null/misaligned pointer, bad size or flag) */
  TB_ENOMEM = -2, /* host allocation failed, or a caller buffer is too small */
  TB_EHIP = -3,   /* a HIP runtime call or kernel launch failed */
  TB_ERANGE = -4, /* data out of range (token >= V, blank in a phrase, ...) */
  TB_EIO = -5     /* a file could not be opened, read or written */
};

enum { TB_F32 = 0, TB_BF16 = 1 };                     /* logit element type */
enum { TB_COMMIT = 0, TB_PURE_POTENTIAL = 1 };        /* potential reading   */
/*
 * Special state values (graph states are otherwise >= 0):
 *   TB_STATE_NONE     model -1: the stream is not biased.
 *   TB_STATE_INVALID  the stream's model id or carried state was out of range
 *                     for the arena: the stream is decoded without biasing.
 *   TB_STATE_TIMEOUT  a bounded wait inside a greedy step kernel gave up (the
 *                     waves of one workgroup hand states to each other; this
 *                     should never happen and indicates a fault). The rows
 *                     written as TB_STATE_TIMEOUT, and the stream's later
 *                     rows, are unreliable. The state is sticky: a carried
 *                     TB_STATE_TIMEOUT makes later calls decode that stream
 *                     without biasing and write TB_STATE_TIMEOUT again, until
 *                     tb_reset_stream or tb_init_states restarts it.
 */
enum { TB_STATE_NONE = -1, TB_STATE_INVALID = -2, TB_STATE_TIMEOUT = -3 };

/* Host-side compiled graphs of all models (library owned). */
typedef struct tb_graphs tb_graphs;

/*
 * Layout of the device arena image: one contiguous byte buffer holding the
 * merged multi-model storage of Sec. II-B (all models' state tensors
 * concatenated, a per-model table of offsets, and per-model root rows).
 * All offsets are in bytes from the start of the buffer, 256-byte aligned.
 *
 *   model_off   int32[n_models]   first global state index of each model
 *   model_n     int32[n_models]   number of states of each model
 *   first_child int32[n_states]   local id of the first child (children are
 *                                 contiguous ids, labels strictly ascending)
 *   n_child     int32[n_states]   number of children
 *   link        int32[n_states]   suffix-link target, local id (< own id)
 *   label       int32[n_states]   class of the arc into the state (root: -1)
 *   phi         float[n_states]   potential phi (pending score)
 *   psi         float[n_states]   phi + end bonus E: a step into state x from
 *                                 state s scores psi[x] - phi[s]
 *   root_psi    float[n_models*(V+1)]  psi of the root move of every token
 *                                      (blank column: 0)
 *   root_dst    int32[n_models*(V+1)]  local state of the root move of every
 *                                      token (blank column: 0)
 *   class_map   int32[V+1]        token -> case class (blank: -1)
 *   cls_ptr     int32[V+1]        CSR over classes: members of class c are
 *   cls_tok     int32[V]          cls_tok[cls_ptr[c] .. cls_ptr[c+1]-1], ascending
 *   arc_mem     uint32[2*n_states] the class on the arc into every state with
 *                                 its first three members m0 <= m1 <= m2
 *                                 (repeating the last when the class is
 *                                 smaller): word 0 = m0 | m1 << 16, word 1 =
 *                                 m2 | class << 16 | (more than three
 *                                 members ? 1 << 31 : 0); roots: 0, 0
 *                                 (token ids and classes below 2^15)
 *   value_tab   float[n_models*512]  per model the distinct psi values
 *                                 (entries 0..255, ascending) and the
 *                                 distinct phi values (entries 256..511)
 *   state_rec   uint32[3*n_states]  a packed record of every state x:
 *                 word 0 = first_child & 0xffff | min(n_child, 255) << 16 |
 *                          psi index << 24
 *                 word 1 = link & 0xffff | cls_ptr[label] << 16 (the first
 *                          member of the arc class in cls_tok; roots: 0)
 *                 word 2 = class size (<= 255) | phi index << 8 |
 *                          label << 16 (15 bits; roots: 0) | flag << 31
 *               The flag is set when a field does not fit (first child, link
 *               or class size >= 2^16 / 255, n_child >= 255, or more than
 *               256 distinct psi or phi values in the model); the record is
 *               then not used and the plain arrays above are read instead.
 */
typedef struct {
  int64_t total_bytes;
  int32_t n_models;
  int32_t v_plus_blank;
  int64_t n_states; /* sum over models */
  int64_t off_model_off, off_model_n;
  int64_t off_first_child, off_n_child, off_link, off_label, off_phi, off_psi;
  int64_t off_root_psi, off_root_dst;
  int64_t off_class_map, off_cls_ptr, off_cls_tok;
  int64_t off_arc_mem;
  int32_t max_children;  /* largest out-degree of any state */
  int32_t max_depth;     /* deepest state (phrase length) */
  int32_t max_override;  /* most tokens any state overrides: the members of the
                            classes of the children along its suffix chain */
  int64_t off_value_tab, off_state_rec;
} tb_arena_layout;

/* A device-resident arena: the layout plus the device address of the image. */
typedef struct {
  const void* base; /* device pointer to tb_arena_layout.total_bytes bytes */
  tb_arena_layout layout;
} tb_arena;

/*
 * tb_compile_graphs — compile per-stream phrase lists into merged storage
 * (Sec. II-B "per-stream context-biasing model"; case-insensitive graph of
 * Sec. II-A: every token is replaced by its case class, so one arc accepts
 * every case variant).
 *
 *   n_models          number of phrase lists (models), >= 1
 *   model_phrase_ptr  host int64[n_models+1], CSR over phrases
 *   phrase_tok_ptr    host int64[n_phrases+1], CSR over tokens
 *   phrase_tokens     host int32[phrase_tok_ptr[n_phrases]]; ids in [0, V)
 *   token_w           host float[n_models], score per matched token (w)
 *   end_bonus         host float[n_models], end-of-phrase bonus
 *   scale             host float[n_models] or NULL (= 1): the per-model
 *                     boosting weight, folded into phi and psi
 *   class_map         host int32[v_plus_blank]; class of every token (a token
 *                     id in [0, V)), class_map[V] must be -1
 *   v_plus_blank      V + 1, in [2, 32768]
 *   semantics         TB_COMMIT (default reading) or TB_PURE_POTENTIAL
 *   n_threads         host threads to use (<= 0: hardware concurrency)
 *   out               receives the library-owned result; free with
 *                     tb_graphs_free
 *
 * An empty list gives a root-only graph (state 0, zero boost). Duplicate
 * phrases (after case folding) are merged. Errors: TB_EINVAL (null pointers,
 * non-monotone CSR, v_plus_blank < 2), TB_ERANGE (token outside [0, V), a
 * token whose class is -1, an empty phrase, a class id outside [0, V),
 * v_plus_blank > 32768), TB_ENOMEM.
 */
int tb_compile_graphs(int32_t n_models, const int64_t* model_phrase_ptr,
                      const int64_t* phrase_tok_ptr, const int32_t* phrase_tokens,
                      const float* token_w, const float* end_bonus, const float* scale,
                      const int32_t* class_map, int32_t v_plus_blank, int32_t semantics,
                      int32_t n_threads, tb_graphs** out);

/* Layout (sizes and offsets) of the arena image of g. */
int tb_graphs_layout(const tb_graphs* g, tb_arena_layout* out);

/* Copy the arena image into host memory dst (bytes >= layout.total_bytes). */
int tb_graphs_host_image(const tb_graphs* g, void* dst, int64_t bytes);

/*
 * tb_compile_variative — per-stream phrase lists written in characters,
 * compiled into the case-insensitive variative BPE graph (Sec. II-A, Fig. 1c
 * and 1e) with the Eq. (1) potentials, as an arena image for the same step
 * calls.
 *
 * The vocabulary is given as pieces: token v (0 <= v < V) spells
 * token_chars[token_char_ptr[v] .. token_char_ptr[v+1]) (at least one
 * character; codes in [0, n_chars)); lower[c] is the lowercase of character
 * c. A token's class is the smallest token id with the same lowercased
 * spelling (the class map of the image; the blank V has class -1). Every
 * character used by a phrase must also be a single-character piece.
 *
 * Per list, the lowercased phrases form a character trie; from every node,
 * every piece class whose lowercased spelling continues the trie is an arc to
 * the node it reaches (a DAG: arcs of different lengths converge), with
 * character-level suffix links. Each phrase's greedy tokenization (longest
 * lowercased piece from the left) carries the score: backbone token k of
 * m_k characters gives its i-th character the share
 * token_w * exp((i+1)^tau) / sum_j exp((j+1)^tau) (float64), the running
 * sum P along the phrase is kept per node (the largest over the phrases
 * through it), and phi/E/psi follow `semantics` with P in place of the token
 * count of tb_compile_graphs. Every arc is one state standing for the node it
 * reaches: the arcs into a node share its child range, potentials and suffix
 * link (the first arc into its longest proper suffix node). Nodes are
 * numbered by increasing length, one length in order of first arc; a node's
 * out-arcs are consecutive in ascending class order; the root is state 0.
 *
 *   model_phrase_ptr, phrase_char_ptr, phrase_chars  CSR as in
 *                     tb_compile_graphs, over character codes
 *   token_w, end_bonus, scale  as in tb_compile_graphs
 *   token_char_ptr    host int64[V+1], token_chars host int32[...]
 *   v_plus_blank      V + 1, in [2, 32768]
 *   lower             host int32[n_chars], values in [0, n_chars)
 *   tau               finite; 0 splits evenly, larger values move the score
 *                     towards the end of each backbone token
 *
 * Errors: TB_EINVAL (null pointers, non-monotone CSR, v_plus_blank < 2,
 * n_chars < 1, tau not finite, unknown semantics), TB_ERANGE (a character
 * outside [0, n_chars), a token without characters, an empty phrase, a
 * phrase character that is not a single-character piece, v_plus_blank >
 * 32768), TB_ENOMEM.
 */
int tb_compile_variative(int32_t n_models, const int64_t* model_phrase_ptr,
                         const int64_t* phrase_char_ptr, const int32_t* phrase_chars,
                         const float* token_w, const float* end_bonus, const float* scale,
                         const int64_t* token_char_ptr, const int32_t* token_chars,
                         int32_t v_plus_blank, const int32_t* lower, int32_t n_chars, float tau,
                         int32_t semantics, int32_t n_threads, tb_graphs** out);

/*
 * Copy the arena image into caller-owned device memory dev_base (bytes >=
 * layout.total_bytes, 256-byte aligned) on stream and fill *out. Returns once
 * the copy has completed (the host graphs may be freed afterwards).
 */
int tb_graphs_upload(const tb_graphs* g, void* dev_base, int64_t bytes, void* hip_stream,
                     tb_arena* out);

void tb_graphs_free(tb_graphs* g);

/*
 * Check a host copy of an arena image for consistency (every index in range,
 * every suffix chain ending at the root, child ranges of non-root states with
 * ascending labels, root rows consistent with the root's children, class
 * member lists and arc member records consistent with the class map). TB_OK
 * or TB_ERANGE.
 */
int tb_validate_image(const void* host_image, const tb_arena_layout* layout);

/*
 * Model caches (Sec. II-B, lifecycle paragraph: precompiled models kept on
 * disk and in host memory, copied into the merged GPU model on demand; the
 * third level, models registered before a session, is tb_register_models).
 *
 * tb_graphs_cache_create — a host-memory cache of compiled models for one
 *   class map (copied). Entries are per model: one phrase list with its
 *   token_w, end_bonus, scale and semantics, compared exactly. When the held
 *   models would exceed capacity_bytes the least recently used are dropped;
 *   a model larger than capacity_bytes is compiled but not kept. Errors:
 *   TB_EINVAL (null pointer, capacity_bytes < 0, v_plus_blank < 2),
 *   TB_ERANGE (a class map tb_compile_graphs rejects), TB_ENOMEM.
 *
 * tb_graphs_cache_compile — tb_compile_graphs over the cache's class map: a
 *   model found in the cache is taken from it, the others are compiled and
 *   added. The result equals tb_compile_graphs' byte for byte. hits (host
 *   int32*, or NULL) receives the number of models taken from the cache.
 *   Calls on one cache may run concurrently (lookups and insertions are
 *   locked; compiles run outside the lock). Errors as tb_compile_graphs;
 *   TB_EINVAL for a null cache.
 *
 * tb_graphs_cache_stats — host int64[5]: hits, misses, models held, bytes
 *   held (estimated), models dropped.
 */
typedef struct tb_graphs_cache tb_graphs_cache;
int tb_graphs_cache_create(const int32_t* class_map, int32_t v_plus_blank,
                           int64_t capacity_bytes, tb_graphs_cache** out);
int tb_graphs_cache_compile(tb_graphs_cache* c, int32_t n_models,
                            const int64_t* model_phrase_ptr, const int64_t* phrase_tok_ptr,
                            const int32_t* phrase_tokens, const float* token_w,
                            const float* end_bonus, const float* scale, int32_t semantics,
                            int32_t n_threads, int32_t* hits, tb_graphs** out);
int tb_graphs_cache_stats(tb_graphs_cache* c, int64_t* stats);
void tb_graphs_cache_free(tb_graphs_cache* c);

/*
 * tb_graphs_save — write compiled graphs (of tb_compile_graphs,
 *   tb_graphs_cache_compile, tb_compile_variative or tb_graphs_load) to the
 *   file at path, in host byte order: a header (format tag, version, the
 *   layout, the image size and its 64-bit FNV-1a checksum), then the arena
 *   image. The file is written under a temporary name and renamed, so a
 *   reader never sees a partial file. Errors: TB_EINVAL (null argument),
 *   TB_EIO (the file cannot be written).
 *
 * tb_graphs_load — read such a file into new graphs (free with
 *   tb_graphs_free). The layout must be the one its counts imply, the
 *   checksum must match, the image must pass tb_validate_image, and the
 *   layout's max_children and max_override must equal the image's. Errors:
 *   TB_EINVAL (null argument), TB_EIO (missing or unreadable file),
 *   TB_ERANGE (not a graphs file, another version, wrong size, checksum or
 *   content), TB_ENOMEM.
 */
int tb_graphs_save(const tb_graphs* g, const char* path);
int tb_graphs_load(const char* path, tb_graphs** out);

/*
 * tb_init_states — start B streams (Sec. II-B: each stream carries a model id
 * and a state; Sec. II-C: beam scores are carried across chunks).
 *
 *   model_ids  device int32[B]
 *   states     device int32[B*K] out: 0 for a model in range, -1 for -1,
 *              TB_STATE_INVALID for an out-of-range id
 *   scores     device float[B*K] out, or NULL: beam scores [0, -inf, ...]
 */
int tb_init_states(const tb_arena* a, int32_t B, int32_t K, const int32_t* model_ids,
                   int32_t* states, float* scores, void* hip_stream);

/*
 * tb_boost_step_greedy — T boosted greedy steps for B streams (Sec. II-B
 * fused scoring operation, with label selection of greedy Transducer
 * decoding). For step t and stream b with state s and row z = logits[t,b,:]:
 *
 *   key[v] = z[v] + psi[delta(s, class v)]   (v < V; delta = suffix-link move)
 *   key[V] = z[V] + phi[s]                   (blank keeps the state)
 *   v*     = lowest index of the largest key
 *   score  = (z[v*] - lse(z)) + (psi[delta] - phi[s])   (0 boost for blank)
 *
 *   logits     device, element type dtype, row (t,b) at (t*B + b)*row_stride
 *              elements; row_stride >= V+1; 4-byte (f32) / 2-byte (bf16) aligned
 *   model_ids  device int32[B]
 *   states     device int32[B], in: carried state, out: state after step T-1
 *   out_tok, out_state  device int32[T*B];  out_score device float[T*B]
 *
 * T = 0 is a no-op that touches no buffer (logits and outputs may be NULL).
 * Results do not depend on how the T steps are split into calls. Log-softmax here is float32 (|error| well below 1e-5); selection
 * does not depend on it.
 */
int tb_boost_step_greedy(const tb_arena* a, const void* logits, int32_t dtype, int32_t T,
                         int32_t B, int64_t row_stride, const int32_t* model_ids,
                         int32_t* states, int32_t* out_tok, int32_t* out_state,
                         float* out_score, void* hip_stream);

/*
 * tb_boost_step_beam — T boosted beam steps for B streams of K hypotheses
 * (Sec. II-C streaming beam search; K <= TB_MAX_BEAM). Hypothesis k of
 * stream b reads row logits[t,b,k,:] (row index (t*B + b)*K + k) and has
 * state s_k and accumulated score S_k:
 *
 *   lse_k   = log-sum-exp of the row, float64 sum and log, rounded to float32
 *   c_k     = (S_k - lse_k) - phi[s_k]
 *   cand    = c_k + key_k[v]          (key as in the greedy step)
 *   the K largest cand over flat index k*(V+1)+v are kept, sorted descending,
 *   ties to the lowest flat index; slot j takes parent k_j, token v_j, state
 *   delta(s_{k_j}, class v_j) (blank: s_{k_j}) and S_j = cand_j.
 *
 *   states, scores  device [B*K] in/out (carry)
 *   out_tok, out_parent, out_state  device int32[T*B*K]
 *   out_step (the step's log-prob plus boost), out_cum (S)  device float[T*B*K]
 *
 * T = 0 is a no-op that touches no buffer (they may be NULL).
 */
enum { TB_MAX_BEAM = 32 }; /* the paper's beam search uses 32 hypotheses */
int tb_boost_step_beam(const tb_arena* a, const void* logits, int32_t dtype, int32_t T,
                       int32_t B, int32_t K, int64_t row_stride, const int32_t* model_ids,
                       int32_t* states, float* scores, int32_t* out_tok, int32_t* out_parent,
                       int32_t* out_state, float* out_step, float* out_cum, void* hip_stream);

/*
 * Streaming beam search with hypothesis recombination and a flattened
 * hypothesis tree (Sec. II-C: finalized hypotheses are stored in a flattened
 * tree with their accumulated scores and carried across chunks, where they are
 * continued, merged and pruned).
 *
 * A hypothesis is its label sequence (the non-blank tokens it emitted). Each
 * slot carries a tb_hyp: a 64-bit polynomial hash of the sequence (empty: 0;
 * appending label v: h * TB_HASH_MUL + v + 1, modulo 2^64), the hash without
 * the last label, the last label and the tree record of that label. The tree
 * of stream b is tree[(b * tree_cap + r) * 2 + {0, 1}] = (label, parent
 * record) for r < tree_len[b]; a record that does not fit tree_cap is not
 * stored and the slot's node is -2. A node is -1 for the empty sequence.
 */
#define TB_HASH_MUL 0x9E3779B97F4A7C15ull
typedef struct {
  uint64_t hash;        /* hash of the label sequence */
  uint64_t prefix_hash; /* hash of the sequence without its last label (0 if empty) */
  int32_t last;         /* last label, -1 if empty */
  int32_t node;         /* tree record of the last label, -1 if empty, -2 if it did not fit */
} tb_hyp;

/*
 * tb_init_beam_stream — tb_init_states for the streaming beam, plus empty
 * hypotheses: hyps device tb_hyp[B*K] (8-byte aligned) out, tree_len device
 * int32[B] out (0).
 */
int tb_init_beam_stream(const tb_arena* a, int32_t B, int32_t K, const int32_t* model_ids,
                        int32_t* states, float* scores, tb_hyp* hyps, int32_t* tree_len,
                        void* hip_stream);

/*
 * tb_boost_step_beam_stream — tb_boost_step_beam (same arguments and per-step
 * outputs) with the hypothesis carry and tree. With recombine != 0, two
 * candidates of a step with equal label sequences (necessarily slot i extended
 * by the blank and the slot holding i's sequence without its last label,
 * extended by that label; both live) are merged before the K best are taken:
 * the better one in (score, flat index) order keeps its position with score
 * log(exp(a) + exp(b)) (float64, rounded once to float32), the other is
 * dropped. Every kept non-blank extension appends a record (label, parent
 * slot's node) to its stream's tree, in slot order.
 *
 *   hyps      device tb_hyp[B*K] in/out (8-byte aligned), from tb_init_beam_stream
 *   tree      device int32[B * tree_cap * 2] in/out; may be NULL when tree_cap is 0
 *             (no record is stored, nodes are -2)
 *   tree_len  device int32[B] in/out: records stored per stream (a value
 *             outside [0, tree_cap] is read as its nearest bound)
 *   recombine 0: no merging (then the outputs equal tb_boost_step_beam's)
 *
 * Label sequences are compared by their hashes (a collision of two different
 * sequences among one stream's live slots would merge them). K in [1,
 * TB_MAX_BEAM] and K <= V+1, else TB_EINVAL. Concurrent calls on the same
 * carry race.
 */
int tb_boost_step_beam_stream(const tb_arena* a, const void* logits, int32_t dtype, int32_t T,
                              int32_t B, int32_t K, int64_t row_stride, const int32_t* model_ids,
                              int32_t* states, float* scores, tb_hyp* hyps, int32_t* tree,
                              int32_t tree_cap, int32_t* tree_len, int32_t recombine,
                              int32_t* out_tok, int32_t* out_parent, int32_t* out_state,
                              float* out_step, float* out_cum, void* hip_stream);

/*
 * tb_reset_stream — give stream b (0 <= b < B) a new model id (Sec. II-B:
 * lists are added and removed as streams start and finish) and restart its
 * carry: model id new_model_id in [-1, n_models), states 0 (or -1), scores
 * [0, -inf, ...] (scores may be NULL). model_ids is device int32[B], states
 * and scores device [B*K]. Only stream b's entries are written.
 */
int tb_reset_stream(const tb_arena* a, int32_t B, int32_t b, int32_t new_model_id, int32_t K,
                    int32_t* model_ids, int32_t* states, float* scores, void* hip_stream);

/*
 * Model lifecycle (Sec. II-B: per-stream lists are added and removed as
 * streams start and finish; adding appends a model's tensors and records its
 * offsets, removing marks its id inactive and shifts the later ranges left;
 * stream-facing model ids are kept apart from the physical offsets).
 *
 * A registry is an arena with free capacity: tb_compile_graphs' image layout
 * sized for max_models model slots (the stable ids 0..max_models-1) and
 * max_states states, in caller-owned device memory. tb_registry_arena gives
 * the tb_arena that step calls take; a free or removed id decodes like an
 * out-of-range one (no biasing, states TB_STATE_INVALID), so streams on a
 * removed model should be reset. Lifecycle calls and step calls on one
 * registry must be ordered on one stream (the step calls read the model
 * table and the moved ranges). The registry handle is host memory owned by
 * the library (tb_registry_free); calls that take it must not overlap in
 * time (the lifecycle calls update its host copy of the model table and its
 * staging buffer), so host threads that share one registry serialise them.
 *
 * tb_registry_layout — layout (and total_bytes) of a registry's device
 *   arena; max_models >= 1, max_states in [max_models, 2^31), v_plus_blank
 *   in [2, 32768]. TB_EINVAL otherwise.
 * tb_registry_create — start an empty registry (every id free) in dev_base
 *   (device, 256-byte aligned, >= total_bytes, else TB_EINVAL / TB_ENOMEM)
 *   with the class map of every model it will hold (host int32[v_plus_blank],
 *   as tb_compile_graphs; TB_ERANGE when invalid). Returns once the tables
 *   are on the device.
 * tb_registry_model — device range of id: first state and state count (0:
 *   free). TB_ERANGE for an id outside [0, max_models).
 * tb_register_models — add every model of g (compiled by tb_compile_graphs
 *   with the same class map and v_plus_blank, else TB_EINVAL) at the end of
 *   the used states, under the lowest free ids, written to ids (host
 *   int32[number of models of g]). TB_ENOMEM when ids or states run out
 *   (nothing is changed then). Returns once the copies are done (g may be
 *   freed afterwards).
 * tb_unregister_workspace_bytes — device scratch tb_unregister_model needs
 *   for id (44 bytes per state after the model); -1 for a free id.
 * tb_unregister_model — remove id: its states are filled by the later ones,
 *   moved left by a compaction kernel through workspace (device, 4-byte
 *   aligned, >= tb_unregister_workspace_bytes, else TB_ENOMEM before any
 *   launch), and the model table is rebased on the device. Asynchronous on
 *   hip_stream; the workspace is free again once the stream has passed the
 *   call. TB_EINVAL for a free id.
 */
typedef struct tb_registry tb_registry;
int tb_registry_layout(int32_t max_models, int64_t max_states, int32_t v_plus_blank,
                       tb_arena_layout* out);
int tb_registry_create(int32_t max_models, int64_t max_states, const int32_t* class_map,
                       int32_t v_plus_blank, void* dev_base, int64_t bytes, void* hip_stream,
                       tb_registry** out);
int tb_registry_arena(const tb_registry* r, tb_arena* out);
int tb_registry_model(const tb_registry* r, int32_t id, int64_t* first_state, int32_t* n_states);
int64_t tb_registry_used_states(const tb_registry* r); /* states in use; -1 for NULL */
int tb_register_models(tb_registry* r, const tb_graphs* g, int32_t* ids, void* hip_stream);
int64_t tb_unregister_workspace_bytes(const tb_registry* r, int32_t id);
int tb_unregister_model(tb_registry* r, int32_t id, void* workspace, int64_t workspace_bytes,
                        void* hip_stream);
void tb_registry_free(tb_registry* r);

/*
 * tb_unregister_model_noalloc — tb_unregister_model for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the compaction goes through a scratch
 * array the library holds in device memory, 32 MiB on every device it runs
 * on, kept until the process ends. Removing a model whose later states take
 * more than 32 MiB of records (44 bytes per state) is rejected with TB_ENOMEM
 * before any launch. Every call on one device shares that device's scratch:
 * calls that overlap on one device (different streams, or threads) race;
 * order them. Otherwise as tb_unregister_model (allocates nothing).
 */
int tb_unregister_model_noalloc(tb_registry* r, int32_t id, void* hip_stream);

/* Message of the last failed call on this thread ("" if none). */
const char* tb_last_error(void);

/*
 * Test hooks (not for production use). They change process-wide settings
 * that later step calls read; calls that overlap a change see either value.
 *
 * tb_debug_select_kernels — force a kernel family so that tests can compare
 * every path: greedy 0 = automatic choice, 1 = the reference kernel (one
 * workgroup per stream, any V); beam 0 = automatic, 1 = the reference kernel,
 * 2 = automatic but never the helper-wave kernel. TB_EINVAL for other values.
 *
 * tb_debug_set_spin_limit — polls after which the greedy hand-off wait (the
 * waves of a workgroup pass exact states in order) gives up and writes
 * TB_STATE_TIMEOUT; 0 restores the default (2^26, never reached in normal
 * operation). A limit of 1 lets a test force the timeout path from the host;
 * the kernel still ends normally.
 */
int tb_debug_select_kernels(int32_t greedy, int32_t beam);
int tb_debug_set_spin_limit(uint32_t polls);

/*
 * tb_debug_launch_empty — enqueue a kernel that does nothing, with grid
 * workgroups of block threads (<= 1024) and lds_bytes of dynamic LDS (<= 160
 * KiB), on hip_stream: what a step kernel's launch of that shape costs by
 * itself (the benchmark's launch floor). TB_EINVAL for other shapes.
 */
int tb_debug_launch_empty(int32_t grid, int32_t block, int32_t lds_bytes, void* hip_stream);

#ifdef __cplusplus
}
#endif
#endif /* TBIAS_H */
