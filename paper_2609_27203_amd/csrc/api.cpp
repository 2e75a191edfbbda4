// extern "C" entry points declared in include/xlh.h.
#include <algorithm>
#include <cstring>
#include <mutex>

#include "engine.h"

using namespace xlh;

namespace {
constexpr size_t PINNED_BYTES = CTL_BYTES;
constexpr int STATIC_MAX_DEVICES = 64;
}  // namespace

struct xl_context : Context {
  bool static_ws = false;  // the arena is the device's static workspace (xl_context_create_static)
  alignas(64) unsigned char ctl[PINNED_BYTES];  // control block of a static context (no pinned allocation)
};
struct xl_relation : Relation {};
struct xl_program : Program {};

// Workspace of the allocation-free contexts: one copy per device the library
// runs on, held until the process ends.  In host code `scratch` names a host
// stand-in, never the device memory: its device address on each device comes
// from hipGetSymbolAddress (with that device current) and is kept below.
static __device__ __align__(256) unsigned char scratch[XL_STATIC_WORKSPACE_BYTES];

namespace {
std::mutex g_static_mu;
void* g_static_ptr[STATIC_MAX_DEVICES] = {};  // device address of `scratch`, per device
bool g_static_held[STATIC_MAX_DEVICES] = {};  // a live static context uses that device's copy
}  // namespace

extern "C" {

const char* xl_status_string(xl_status s) {
  switch (s) {
    case XL_OK: return "XL_OK";
    case XL_INVALID_ARGUMENT: return "XL_INVALID_ARGUMENT";
    case XL_TYPE_MISMATCH: return "XL_TYPE_MISMATCH";
    case XL_UNSUPPORTED: return "XL_UNSUPPORTED";
    case XL_RESOURCE_EXHAUSTED: return "XL_RESOURCE_EXHAUSTED";
    case XL_CAPACITY_EXCEEDED: return "XL_CAPACITY_EXCEEDED";
    case XL_CONVERGENCE_FAILURE: return "XL_CONVERGENCE_FAILURE";
    case XL_DEVICE_ERROR: return "XL_DEVICE_ERROR";
    case XL_PARSE_ERROR: return "XL_PARSE_ERROR";
  }
  return "unknown status";
}

xl_status xl_context_create(int device, void* hip_stream, void* workspace, size_t workspace_bytes,
                            xl_context** out) {
  if (!out) return XL_INVALID_ARGUMENT;
  auto* c = new xl_context();
  c->device = device;
  if (device >= 0) {
    if (!workspace || workspace_bytes < (1u << 20)) {
      delete c;
      return XL_INVALID_ARGUMENT;
    }
    if (hipSetDevice(device) != hipSuccess) {
      delete c;
      return XL_DEVICE_ERROR;
    }
    c->stream = (hipStream_t)hip_stream;
    c->arena.init((char*)workspace, workspace_bytes);
    if (hipHostMalloc(&c->pinned, PINNED_BYTES, hipHostMallocDefault) != hipSuccess) {
      delete c;
      return XL_DEVICE_ERROR;
    }
    c->dcounters = (unsigned long long*)c->arena.alloc(8 * CNT_N);
    c->dcheck = (unsigned long long*)c->arena.alloc(8);
  }
  *out = c;
  return XL_OK;
}

xl_status xl_context_create_static(int device, void* hip_stream, xl_context** out) {
  if (!out || device < 0 || device >= STATIC_MAX_DEVICES) return XL_INVALID_ARGUMENT;
  if (hipSetDevice(device) != hipSuccess) return XL_DEVICE_ERROR;
  std::lock_guard<std::mutex> lock(g_static_mu);
  if (g_static_held[device]) return XL_RESOURCE_EXHAUSTED;
  if (!g_static_ptr[device]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return XL_DEVICE_ERROR;
    g_static_ptr[device] = p;
  }
  auto* c = new xl_context();
  c->device = device;
  c->stream = (hipStream_t)hip_stream;
  c->static_ws = true;
  c->pinned = c->ctl;
  c->arena.init((char*)g_static_ptr[device], XL_STATIC_WORKSPACE_BYTES);
  c->dcounters = (unsigned long long*)c->arena.alloc(8 * CNT_N);
  c->dcheck = (unsigned long long*)c->arena.alloc(8);
  g_static_held[device] = true;
  *out = c;
  return XL_OK;
}

xl_status xl_context_set_option(xl_context* c, const char* key, int64_t value) {
  if (!c || !key) return XL_INVALID_ARGUMENT;
  if (!strcmp(key, "hash_min_log2")) {
    if (value < 10 || value > 34) return c->fail(XL_INVALID_ARGUMENT, "hash_min_log2 must be in [10, 34]");
    c->hash_min_log2 = (int)value;
    return XL_OK;
  }
  if (!strcmp(key, "index_mode")) {
    if (value < 0 || value > 2) return c->fail(XL_INVALID_ARGUMENT, "index_mode must be 0, 1 or 2");
    c->index_mode = (int)value;
    return XL_OK;
  }
  if (!strcmp(key, "pull_ratio")) {
    if (value < 0 || value > 1024) return c->fail(XL_INVALID_ARGUMENT, "pull_ratio must be in [0, 1024]");
    c->pull_ratio = (int)value;
    return XL_OK;
  }
  if (!strcmp(key, "index_cache_mb")) {
    if (value < 0 || value > ((int64_t)1 << 20)) return c->fail(XL_INVALID_ARGUMENT, "index_cache_mb must be in [0, 2^20]");
    c->index_cache_bytes = (size_t)value << 20;
    if (value == 0)
      while (!c->icache.empty()) c->icache_drop(c->icache.front().rel, false);
    return XL_OK;
  }
  if (!strcmp(key, "batched_rounds")) {
    if (value < 0 || value > 64) return c->fail(XL_INVALID_ARGUMENT, "batched_rounds must be in [0, 64]");
    c->batched_rounds = (int)value;
    return XL_OK;
  }
  if (!strcmp(key, "gather_rounds")) {
    if (value < 0 || value > 2) return c->fail(XL_INVALID_ARGUMENT, "gather_rounds must be 0, 1 or 2");
    c->gather_rounds = (int)value;
    return XL_OK;
  }
  if (!strcmp(key, "product_joins")) {
    if (value != 0 && value != 1) return c->fail(XL_INVALID_ARGUMENT, "product_joins must be 0 or 1");
    c->product_joins = (int)value;
    return XL_OK;
  }
  if (!strcmp(key, "wcoj_shorter")) {
    if (value != 0 && value != 1) return c->fail(XL_INVALID_ARGUMENT, "wcoj_shorter must be 0 or 1");
    c->wcoj_shorter = (int)value;
    return XL_OK;
  }
  if (!strcmp(key, "frontier_resident")) {
    if (value != 0 && value != 1) return c->fail(XL_INVALID_ARGUMENT, "frontier_resident must be 0 or 1");
    c->frontier_resident = (int)value;
    return XL_OK;
  }
  if (!strcmp(key, "dense_tiles")) {
    if (value < -1 || value > 4096) return c->fail(XL_INVALID_ARGUMENT, "dense_tiles must be in [-1, 4096]");
    c->dense_tiles = (int)value;
    return XL_OK;
  }
  if (!strcmp(key, "profile")) {
    if (value < 0 || value > 1) return c->fail(XL_INVALID_ARGUMENT, "profile must be 0 or 1");
    c->profile = (int)value;
    return XL_OK;
  }
  return c->fail(XL_INVALID_ARGUMENT, std::string("unknown option '") + key + "'");
}

xl_status xl_relation_create(xl_context* c, const char* name, int arity, const xl_type* cols,
                             int64_t max_rows, xl_relation** out) {
  if (!c || !name || !cols || !out) return XL_INVALID_ARGUMENT;
  if (arity < 1 || arity > XL_MAX_ARITY) return c->fail(XL_INVALID_ARGUMENT, "arity must be 1..4");
  if (max_rows < 0) return c->fail(XL_INVALID_ARGUMENT, "negative max_rows");
  if (!*name || !(islower((unsigned char)name[0])))
    return c->fail(XL_INVALID_ARGUMENT, "relation names start with a lower-case letter");
  for (const char* p = name; *p; ++p)
    if (!isalnum((unsigned char)*p) && *p != '_') return c->fail(XL_INVALID_ARGUMENT, "bad relation name");
  if (c->find(name)) return c->fail(XL_INVALID_ARGUMENT, std::string("relation '") + name + "' already exists");
  for (int j = 0; j < arity; ++j)
    if (cols[j] < XL_I32 || cols[j] > XL_BOOL) return c->fail(XL_INVALID_ARGUMENT, "unknown column type");
  auto* r = new xl_relation();
  r->ctx = c;
  r->name = name;
  r->arity = arity;
  for (int j = 0; j < arity; ++j) {
    r->ltypes[j] = (uint8_t)cols[j];
    r->types[j] = phys_type(cols[j]);
  }
  r->max_rows = max_rows;
  c->rels.push_back(r);
  *out = r;
  return XL_OK;
}

xl_status xl_relation_load(xl_relation* r, const void* const* cols, int64_t nrows, int cols_on_device) {
  if (!r) return XL_INVALID_ARGUMENT;
  return relation_load(r, cols, nrows, cols_on_device);
}

xl_status xl_relation_clear(xl_relation* r) {
  if (!r) return XL_INVALID_ARGUMENT;
  return relation_clear(r);
}

xl_status xl_relation_size(const xl_relation* r, int64_t* out_rows) {
  if (!r || !out_rows) return XL_INVALID_ARGUMENT;
  *out_rows = r->nrows;
  return XL_OK;
}

xl_status xl_relation_read(const xl_relation* r, void* const* cols, int64_t capacity_rows, int64_t* out_rows,
                           int cols_on_device) {
  if (!r) return XL_INVALID_ARGUMENT;
  if (r->ctx->device < 0) return r->ctx->fail(XL_INVALID_ARGUMENT, "planning-only context holds no data");
  return relation_read(r, cols, capacity_rows, out_rows, cols_on_device);
}

xl_status xl_rule_compile(xl_context* c, const char* text, xl_program** out) {
  if (!c || !text || !out) return XL_INVALID_ARGUMENT;
  Program* p = nullptr;
  xl_status s = compile_program(c, text, &p);
  if (s != XL_OK) return s;
  auto* xp = new xl_program();
  static_cast<Program&>(*xp) = std::move(*p);
  delete p;
  c->progs.push_back(xp);
  *out = xp;
  return XL_OK;
}

xl_status xl_program_explain(const xl_program* p, char* buf, size_t cap, size_t* needed) {
  if (!p) return XL_INVALID_ARGUMENT;
  std::string s = explain_program(p);
  if (needed) *needed = s.size() + 1;
  if (buf && cap) {
    size_t n = std::min(cap - 1, s.size());
    memcpy(buf, s.data(), n);
    buf[n] = 0;
  }
  return XL_OK;
}

xl_status xl_fixpoint_run(xl_program* p, int64_t max_iterations, xl_fixpoint_stats* out_stats) {
  if (!p) return XL_INVALID_ARGUMENT;
  xl_fixpoint_stats local;
  xl_fixpoint_stats* st = out_stats ? out_stats : &local;
  if (p->ctx->device >= 0 && hipSetDevice(p->ctx->device) != hipSuccess) return XL_DEVICE_ERROR;
  return run_program(p, max_iterations, st);
}

const char* xl_last_error(const xl_context* c) { return c ? c->err.c_str() : "null context"; }

void xl_program_destroy(xl_program* p) {
  if (!p) return;
  auto& v = p->ctx->progs;
  v.erase(std::remove(v.begin(), v.end(), static_cast<Program*>(p)), v.end());
  delete p;
}

void xl_relation_destroy(xl_relation* r) {
  if (!r) return;
  Context* c = r->ctx;
  if (c->device >= 0) {
    relation_free_storage(r);
    c->icache_drop(r, false);
  }
  c->rels.erase(std::remove(c->rels.begin(), c->rels.end(), static_cast<Relation*>(r)), c->rels.end());
  delete r;
}

void xl_context_destroy(xl_context* c) {
  if (!c) return;
  if (c->device >= 0 && c->stream) (void)hipStreamSynchronize(c->stream);
  for (Program* p : c->progs) delete static_cast<xl_program*>(p);
  for (Relation* r : c->rels) delete static_cast<xl_relation*>(r);
  if (c->static_ws) {
    std::lock_guard<std::mutex> lock(g_static_mu);
    g_static_held[c->device] = false;
  } else if (c->pinned) {
    (void)hipHostFree(c->pinned);
  }
  delete c;
}

}  // extern "C"
