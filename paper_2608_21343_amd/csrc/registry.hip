// Model lifecycle on a device arena with free capacity (Sec. II-B: models are
// added by appending their state tensors and recording their offsets, and
// removed by marking the id inactive and shifting the later state ranges left
// to fill the gap; stream-facing model ids stay stable while offsets move).
//
// The arena has the image layout of tb_compile_graphs, sized for max_models
// model slots and max_states states. A model's state records use model-local
// ids only (children, suffix links), so moving its range changes nothing but
// its offset in the model table. Per-model rows (root row, value table) are
// indexed by the stable id and never move.
#include <algorithm>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "device.hpp"
#include "internal.hpp"

struct tb_registry {
  tb_arena arena;                  // base + layout (capacities; maxima over models ever added)
  int32_t max_models = 0;
  int64_t max_states = 0;
  int64_t used = 0;                // states in use: [0, used)
  std::vector<int32_t> off, n;     // host copy of the model table (n == 0: free id)
  std::vector<int32_t> class_map;  // the arena's class map
  // pinned host staging of tb_register_models (grown on demand): copies from
  // it run asynchronously, without the per-copy staging of pageable memory
  unsigned char* stage = nullptr;
  size_t stage_bytes = 0;
  ~tb_registry() {
    if (stage) (void)hipHostFree(stage);
  }
};

namespace tbias {
namespace {

// Per-state arrays of the image: byte offset in the layout and 32-bit words
// per state.
struct StateArray {
  int64_t off;
  int32_t words;
};

inline int state_arrays(const tb_arena_layout& L, StateArray* a) {
  a[0] = {L.off_first_child, 1};
  a[1] = {L.off_n_child, 1};
  a[2] = {L.off_link, 1};
  a[3] = {L.off_label, 1};
  a[4] = {L.off_phi, 1};
  a[5] = {L.off_psi, 1};
  a[6] = {L.off_arc_mem, 2};
  a[7] = {L.off_state_rec, 3};
  return 8;
}
constexpr int kStateWords = 11;  // words per state over all per-state arrays

constexpr int kMaxSegs = 8;
struct Segs {
  const uint32_t* src[kMaxSegs];
  uint32_t* dst[kMaxSegs];
  int64_t words[kMaxSegs];
  int32_t n;
};

// Copies up to eight word ranges (no range overlaps another's destination):
// grid row y copies range y, grid-stride, four words per thread in flight.
__global__ void copy_segments_kernel(Segs S) {
  const int k = blockIdx.y;
  if (k >= S.n) return;
  const uint32_t* __restrict__ src = S.src[k];
  uint32_t* __restrict__ dst = S.dst[k];
  const int64_t words = S.words[k];
  const int64_t step = (int64_t)gridDim.x * blockDim.x;
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 3 * step < words; i += 4 * step) {
    const uint32_t a = src[i], b = src[i + step], c = src[i + 2 * step], d = src[i + 3 * step];
    dst[i] = a;
    dst[i + step] = b;
    dst[i + 2 * step] = c;
    dst[i + 3 * step] = d;
  }
  for (; i < words; i += step) dst[i] = src[i];
}

// The model table after removing the model at [off, off + n): the removed id
// becomes free, later ranges move left by n.
__global__ void rebase_kernel(int32_t* model_off, int32_t* model_n, int32_t max_models,
                              int32_t id, int32_t off, int32_t n) {
  const int32_t j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= max_models) return;
  if (j == id) {
    model_off[j] = 0;
    model_n[j] = 0;
  } else if (model_n[j] > 0 && model_off[j] > off) {
    model_off[j] -= n;
  }
}

int hip_fail(hipError_t e, const char* what) {
  return fail(TB_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

hipError_t launch_copy(const Segs& S, hipStream_t st) {
  int64_t most = 0;
  for (int k = 0; k < S.n; ++k) most = std::max(most, S.words[k]);
  if (most == 0) return hipSuccess;
  const int threads = 256;
  int64_t blocks = (most + 4 * threads - 1) / (4 * threads);
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(copy_segments_kernel, dim3((uint32_t)blocks, (uint32_t)S.n), dim3(threads),
                     0, st, S);
  return hipGetLastError();
}

unsigned char* dev_bytes(const tb_registry* r) {
  return static_cast<unsigned char*>(const_cast<void*>(r->arena.base));
}

// Scratch of tb_unregister_model_noalloc: one copy on every device the
// library runs on, held until the process ends, shared by every call on that
// device. Host code never uses the array's name as an address: the device
// address comes from hipGetSymbolAddress, once per device.
constexpr int64_t kNoAllocScratchBytes = int64_t(32) << 20;
static __device__ __align__(256) uint32_t scratch[kNoAllocScratchBytes / 4];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

// Removal of a registered model with a given scratch buffer (at least
// tb_unregister_workspace_bytes): the later states' records go to scratch,
// then back at their new position; the table is rebased on the device.
int registry_remove(tb_registry* r, int32_t id, uint32_t* scratch, int64_t scratch_bytes,
                    hipStream_t st) {
  if (id < 0 || id >= r->max_models || r->n[id] == 0)
    return fail(TB_EINVAL, "model id " + std::to_string(id) + " is not registered");
  const int32_t off = r->off[id], n = r->n[id];
  const int64_t tail = r->used - ((int64_t)off + n);
  const int64_t need = tail * kStateWords * 4;
  if (tail > 0 && (!scratch || scratch_bytes < need))
    return fail(TB_ENOMEM, "workspace of " + std::to_string(scratch_bytes) + " bytes, removing model " +
                               std::to_string(id) + " needs " + std::to_string(need));
  const tb_arena_layout& L = r->arena.layout;
  unsigned char* base = dev_bytes(r);
  if (tail > 0) {
    StateArray a[8];
    const int na = state_arrays(L, a);
    Segs out, back;
    out.n = back.n = na;
    int64_t w0 = 0;
    for (int k = 0; k < na; ++k) {
      uint32_t* arr = reinterpret_cast<uint32_t*>(base + a[k].off);
      const int64_t words = tail * a[k].words;
      out.src[k] = arr + ((int64_t)off + n) * a[k].words;
      out.dst[k] = scratch + w0;
      out.words[k] = words;
      back.src[k] = scratch + w0;
      back.dst[k] = arr + (int64_t)off * a[k].words;
      back.words[k] = words;
      w0 += words;
    }
    hipError_t e = launch_copy(out, st);
    if (e != hipSuccess) return hip_fail(e, "compaction copy-out launch");
    e = launch_copy(back, st);
    if (e != hipSuccess) return hip_fail(e, "compaction copy-back launch");
  }
  const int32_t threads = 256;
  hipLaunchKernelGGL(rebase_kernel, dim3((r->max_models + threads - 1) / threads), dim3(threads),
                     0, st, reinterpret_cast<int32_t*>(base + L.off_model_off),
                     reinterpret_cast<int32_t*>(base + L.off_model_n), r->max_models, id, off, n);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "model table rebase launch");
  for (int32_t j = 0; j < r->max_models; ++j)
    if (j != id && r->n[j] > 0 && r->off[j] > off) r->off[j] -= n;
  r->off[id] = 0;
  r->n[id] = 0;
  r->used -= n;
  return TB_OK;
}

}  // namespace tbias

using namespace tbias;

extern "C" int tb_registry_layout(int32_t max_models, int64_t max_states, int32_t v_plus_blank,
                                  tb_arena_layout* out) {
  if (!out) return fail(TB_EINVAL, "out is NULL");
  if (max_models < 1) return fail(TB_EINVAL, "max_models must be >= 1");
  if (max_states < max_models || max_states > INT32_MAX)
    return fail(TB_EINVAL, "max_states must be in [max_models, 2^31)");
  if (v_plus_blank < 2 || v_plus_blank > 32768)
    return fail(TB_EINVAL, "v_plus_blank must be in [2, 32768]");
  std::memset(out, 0, sizeof(*out));
  plan_layout(max_models, max_states, v_plus_blank, out);
  return TB_OK;
}

extern "C" int tb_registry_create(int32_t max_models, int64_t max_states, const int32_t* class_map,
                                  int32_t v_plus_blank, void* dev_base, int64_t bytes,
                                  void* hip_stream, tb_registry** out) {
  if (!out) return fail(TB_EINVAL, "out is NULL");
  *out = nullptr;
  if (!class_map || !dev_base) return fail(TB_EINVAL, "NULL argument");
  if (reinterpret_cast<uintptr_t>(dev_base) % 256) return fail(TB_EINVAL, "dev_base not 256-byte aligned");
  tb_arena_layout L;
  int rc = tb_registry_layout(max_models, max_states, v_plus_blank, &L);
  if (rc) return rc;
  if (bytes < L.total_bytes)
    return fail(TB_ENOMEM, "device buffer of " + std::to_string(bytes) + " bytes, the arena needs " +
                               std::to_string(L.total_bytes));
  const int32_t V = v_plus_blank - 1;
  if (class_map[V] != -1) return fail(TB_ERANGE, "class_map[blank] must be -1");
  for (int32_t v = 0; v < V; ++v)
    if (class_map[v] < -1 || class_map[v] >= V)
      return fail(TB_ERANGE, "class_map[" + std::to_string(v) + "] outside [-1, V)");
  auto* r = new (std::nothrow) tb_registry();
  if (!r) return fail(TB_ENOMEM, "host allocation failed");
  r->arena.base = dev_base;
  r->arena.layout = L;
  r->max_models = max_models;
  r->max_states = max_states;
  r->off.assign(max_models, 0);
  r->n.assign(max_models, 0);
  r->class_map.assign(class_map, class_map + v_plus_blank);
  // the model table (every id free) and the class tables
  std::vector<int32_t> zeros(max_models, 0), cp(v_plus_blank, 0), ct(V > 0 ? V : 1, 0);
  class_tables(class_map, V, cp.data(), ct.data());
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  unsigned char* base = static_cast<unsigned char*>(dev_base);
  struct Up { int64_t off; const void* src; size_t bytes; } ups[] = {
      {L.off_model_off, zeros.data(), 4 * (size_t)max_models},
      {L.off_model_n, zeros.data(), 4 * (size_t)max_models},
      {L.off_class_map, class_map, 4 * (size_t)v_plus_blank},
      {L.off_cls_ptr, cp.data(), 4 * (size_t)v_plus_blank},
      {L.off_cls_tok, ct.data(), 4 * (size_t)V},
  };
  for (const Up& u : ups) {
    if (u.bytes == 0) continue;
    hipError_t e = hipMemcpyAsync(base + u.off, u.src, u.bytes, hipMemcpyHostToDevice, st);
    if (e != hipSuccess) { delete r; return hip_fail(e, "hipMemcpyAsync"); }
  }
  hipError_t e = hipStreamSynchronize(st);
  if (e != hipSuccess) { delete r; return hip_fail(e, "hipStreamSynchronize"); }
  *out = r;
  return TB_OK;
}

extern "C" int tb_registry_arena(const tb_registry* r, tb_arena* out) {
  if (!r || !out) return fail(TB_EINVAL, "NULL argument");
  *out = r->arena;
  return TB_OK;
}

extern "C" int tb_registry_model(const tb_registry* r, int32_t id, int64_t* first_state,
                                 int32_t* n_states) {
  if (!r || !first_state || !n_states) return fail(TB_EINVAL, "NULL argument");
  if (id < 0 || id >= r->max_models) return fail(TB_ERANGE, "model id outside [0, max_models)");
  *first_state = r->off[id];
  *n_states = r->n[id];
  return TB_OK;
}

extern "C" int64_t tb_registry_used_states(const tb_registry* r) { return r ? r->used : -1; }

extern "C" int tb_register_models(tb_registry* r, const tb_graphs* g, int32_t* ids,
                                  void* hip_stream) {
  if (!r || !g || !ids) return fail(TB_EINVAL, "NULL argument");
  const tb_arena_layout& G = g->layout;
  tb_arena_layout& L = r->arena.layout;
  if (G.v_plus_blank != L.v_plus_blank)
    return fail(TB_EINVAL, "the graphs were compiled for another vocabulary size");
  const unsigned char* img = g->image.data();
  if (std::memcmp(img + G.off_class_map, r->class_map.data(), 4 * (size_t)L.v_plus_blank) != 0)
    return fail(TB_EINVAL, "the graphs were compiled with another class map");
  // the lowest free ids, and room for the states
  std::vector<int32_t> take;
  for (int32_t j = 0; j < r->max_models && (int32_t)take.size() < G.n_models; ++j)
    if (r->n[j] == 0) take.push_back(j);
  if ((int32_t)take.size() < G.n_models)
    return fail(TB_ENOMEM, std::to_string(G.n_models) + " models to add, " +
                               std::to_string(take.size()) + " free ids");
  if (r->used + G.n_states > r->max_states)
    return fail(TB_ENOMEM, std::to_string(G.n_states) + " states to add, " +
                               std::to_string(r->max_states - r->used) + " free");
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  unsigned char* base = dev_bytes(r);
  const int32_t V1 = L.v_plus_blank;
  // the pieces to copy: (destination offset in the arena, source, bytes);
  // every source is packed into the pinned staging buffer first
  struct Piece {
    int64_t dst;
    const void* src;
    size_t bytes;
  };
  std::vector<Piece> pieces;
  // per-state arrays: every model of g, appended in one range
  StateArray da[8], sa[8];
  const int na = state_arrays(L, da);
  state_arrays(G, sa);
  for (int k = 0; k < na; ++k)
    pieces.push_back({da[k].off + 4 * r->used * da[k].words, img + sa[k].off,
                      4 * (size_t)G.n_states * sa[k].words});
  // per-model rows into the id slots
  const int32_t* g_off = reinterpret_cast<const int32_t*>(img + G.off_model_off);
  const int32_t* g_n = reinterpret_cast<const int32_t*>(img + G.off_model_n);
  for (int32_t i = 0; i < G.n_models; ++i) {
    const int64_t id = take[i];
    pieces.push_back({L.off_root_psi + 4 * id * V1, img + G.off_root_psi + 4 * (int64_t)i * V1,
                      4 * (size_t)V1});
    pieces.push_back({L.off_root_dst + 4 * id * V1, img + G.off_root_dst + 4 * (int64_t)i * V1,
                      4 * (size_t)V1});
    pieces.push_back({L.off_value_tab + 4 * 512 * id, img + G.off_value_tab + 4 * 512 * (int64_t)i,
                      4 * 512});
  }
  std::vector<int32_t> off = r->off, n = r->n;
  for (int32_t i = 0; i < G.n_models; ++i) {
    off[take[i]] = (int32_t)(r->used + g_off[i]);
    n[take[i]] = g_n[i];
  }
  pieces.push_back({L.off_model_off, off.data(), 4 * (size_t)r->max_models});
  pieces.push_back({L.off_model_n, n.data(), 4 * (size_t)r->max_models});
  size_t total = 0;
  for (const Piece& q : pieces) total += (q.bytes + 255) & ~(size_t)255;
  hipError_t e = hipSuccess;
  if (total > r->stage_bytes) {
    if (r->stage) (void)hipHostFree(r->stage);
    r->stage = nullptr;
    r->stage_bytes = 0;
    e = hipHostMalloc(reinterpret_cast<void**>(&r->stage), total, hipHostMallocDefault);
    if (e != hipSuccess) {
      r->stage = nullptr;
      return hip_fail(e, "hipHostMalloc of the registration staging buffer");
    }
    r->stage_bytes = total;
  }
  size_t at = 0;
  for (const Piece& q : pieces) {
    if (q.bytes == 0) continue;
    std::memcpy(r->stage + at, q.src, q.bytes);
    e = hipMemcpyAsync(base + q.dst, r->stage + at, q.bytes, hipMemcpyHostToDevice, st);
    if (e != hipSuccess) break;
    at += (q.bytes + 255) & ~(size_t)255;
  }
  // the staging buffer is reused by the next call: wait for every copy
  const hipError_t es = hipStreamSynchronize(st);
  if (e == hipSuccess) e = es;
  if (e != hipSuccess) return hip_fail(e, "model upload");
  r->off.swap(off);
  r->n.swap(n);
  r->used += G.n_states;
  L.max_children = std::max(L.max_children, G.max_children);
  L.max_depth = std::max(L.max_depth, G.max_depth);
  L.max_override = std::max(L.max_override, G.max_override);
  for (int32_t i = 0; i < G.n_models; ++i) ids[i] = take[i];
  return TB_OK;
}

extern "C" int64_t tb_unregister_workspace_bytes(const tb_registry* r, int32_t id) {
  if (!r || id < 0 || id >= r->max_models || r->n[id] == 0) return -1;
  return (r->used - ((int64_t)r->off[id] + r->n[id])) * 11 * 4;
}

extern "C" int tb_unregister_model(tb_registry* r, int32_t id, void* workspace,
                                   int64_t workspace_bytes, void* hip_stream) {
  if (!r) return fail(TB_EINVAL, "registry is NULL");
  if (workspace && reinterpret_cast<uintptr_t>(workspace) % 4)
    return fail(TB_EINVAL, "workspace not 4-byte aligned");
  return registry_remove(r, id, static_cast<uint32_t*>(workspace), workspace_bytes,
                         static_cast<hipStream_t>(hip_stream));
}

extern "C" int tb_unregister_model_noalloc(tb_registry* r, int32_t id, void* hip_stream) {
  if (!r) return fail(TB_EINVAL, "registry is NULL");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(TB_EINVAL, "device index beyond the scratch table");
  void* ptr = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {  // first call on this device (it is current)
      e = hipGetSymbolAddress(&g_scratch_ptr[dev], HIP_SYMBOL(scratch));
      if (e != hipSuccess) {
        g_scratch_ptr[dev] = nullptr;
        return hip_fail(e, "hipGetSymbolAddress of the scratch array");
      }
    }
    ptr = g_scratch_ptr[dev];
  }
  const int64_t need = tb_unregister_workspace_bytes(r, id);
  if (need > kNoAllocScratchBytes)
    return fail(TB_ENOMEM, "removing model " + std::to_string(id) + " moves " +
                               std::to_string(need) + " bytes of records, beyond the " +
                               std::to_string(kNoAllocScratchBytes) +
                               "-byte scratch of tb_unregister_model_noalloc");
  return registry_remove(r, id, static_cast<uint32_t*>(ptr), kNoAllocScratchBytes,
                         static_cast<hipStream_t>(hip_stream));
}

extern "C" void tb_registry_free(tb_registry* r) { delete r; }
