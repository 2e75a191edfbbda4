// Workspace arena, relation storage, index builds and the semi-naive
// fixpoint driver (host orchestration; every data-plane step is a kernel).
#include <algorithm>
#include <cmath>
#include <cstring>
#include <functional>
#include <memory>

#include "engine.h"
#include "kernels.h"

namespace xlh {

typedef unsigned long long u64;

// Grid cap (blocks of four wavefronts) of the insert-or-improve emission kernels.
constexpr int EMIT_GRID = 2048;
// Rows a wavefront may insert after the load limit is crossed before it
// learns so: its LDS staging buffer (512) plus one 64-item step.
constexpr int64_t WAVE_SLACK = 512 + 64;

// ================================================================== arena
void Arena::init(char* base, size_t size) {
  // every block starts on a 256-B boundary and spans a multiple of 256 B, so
  // kernels may read whole aligned vectors that hold a valid element
  const size_t skip = (256 - (uintptr_t)base % 256) % 256;
  base_ = base + skip;
  size_ = size > skip ? (size - skip) & ~(size_t)255 : 0;
  free_.clear();
  used_.clear();
  if (size_) free_[0] = size_;
  in_use_ = peak_ = 0;
}

void* Arena::alloc(size_t bytes) {
  bytes = (std::max<size_t>(bytes, 1) + 255) & ~(size_t)255;
  for (auto it = free_.begin(); it != free_.end(); ++it) {
    if (it->second < bytes) continue;
    size_t off = it->first, sz = it->second;
    free_.erase(it);
    if (sz > bytes) free_[off + bytes] = sz - bytes;
    used_[off] = bytes;
    in_use_ += bytes;
    peak_ = std::max(peak_, in_use_);
    return base_ + off;
  }
  return nullptr;
}

void Arena::release(void* p) {
  if (!p) return;
  size_t off = (size_t)((char*)p - base_);
  auto it = used_.find(off);
  if (it == used_.end()) return;
  size_t sz = it->second;
  used_.erase(it);
  in_use_ -= sz;
  auto nx = free_.lower_bound(off);
  if (nx != free_.end() && nx->first == off + sz) {
    sz += nx->second;
    free_.erase(nx);
  }
  auto pv = free_.lower_bound(off);
  if (pv != free_.begin()) {
    --pv;
    if (pv->first + pv->second == off) {
      pv->second += sz;
      return;
    }
  }
  free_[off] = sz;
}

size_t Arena::block_size(const void* p) const {
  if (!p) return 0;
  auto it = used_.find((size_t)((const char*)p - base_));
  return it == used_.end() ? 0 : it->second;
}

size_t Arena::largest_free() const {
  size_t m = 0;
  for (auto& kv : free_) m = std::max(m, kv.second);
  return m;
}

// ================================================================== helpers
#define XL_TRY(x)                        \
  do {                                   \
    xl_status _s = (x);                  \
    if (_s != XL_OK) return _s;          \
  } while (0)

#define HIP_TRY(ctx, x)                                                                  \
  do {                                                                                   \
    hipError_t _e = (x);                                                                 \
    if (_e != hipSuccess)                                                                \
      return (ctx)->fail(XL_DEVICE_ERROR, std::string(#x) + ": " + hipGetErrorString(_e)); \
  } while (0)

namespace {

// Arena block released on scope exit unless kept.
struct Buf {
  Context* c = nullptr;
  void* p = nullptr;
  Buf() = default;
  explicit Buf(Context* cc) : c(cc) {}
  Buf(const Buf&) = delete;
  Buf& operator=(const Buf&) = delete;
  ~Buf() { reset(); }
  void reset() {
    if (c && p) c->arena.release(p);
    p = nullptr;
  }
  void* keep() {
    void* q = p;
    p = nullptr;
    return q;
  }
  template <typename T>
  T* as() const {
    return (T*)p;
  }
};

xl_status dalloc(Context* c, size_t bytes, Buf* b, const char* what) {
  b->c = c;
  b->reset();
  b->p = c->arena.alloc(bytes);
  if (!b->p)
    return c->fail(XL_RESOURCE_EXHAUSTED,
                   std::string("workspace exhausted allocating ") + std::to_string(bytes) +
                       " bytes for " + what + " (in use " + std::to_string(c->arena.in_use()) +
                       " of " + std::to_string(c->arena.capacity()) + ", largest free block " +
                       std::to_string(c->arena.largest_free()) + ")");
  return XL_OK;
}

xl_status ctl_read(Context* c, const void* dev, size_t bytes, void* host) {
  if (bytes > CTL_CHECK_OFFSET) return c->fail(XL_DEVICE_ERROR, "control read larger than the control block (internal)");
  HIP_TRY(c, hipMemcpyAsync(c->pinned, dev, bytes, hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  memcpy(host, c->pinned, bytes);
  c->control_bytes += (int64_t)bytes;
  return XL_OK;
}

constexpr int64_t BOUNDS_ONE_MAX = 65536;  // columns this short take one workgroup for their bounds

int bitlen(uint64_t x) {  // bits needed to represent values 0..x
  int b = 0;
  while (x) {
    ++b;
    x >>= 1;
  }
  return b;
}

uint64_t next_pow2(uint64_t x) {
  uint64_t p = 1;
  while (p < x) p <<= 1;
  return p;
}

// Permutation sorting the rows lexicographically (int32 signed, float32
// totalOrder), built as successive stable radix sorts from the last column.
xl_status lex_perm(Context* c, uint32_t* const* cols, const uint8_t* types, int arity, int64_t n,
                   Buf* perm_out) {
  Buf pa, pb, ka, kb, tmp;
  XL_TRY(dalloc(c, (size_t)n * 4, &pa, "sort permutation"));
  XL_TRY(dalloc(c, (size_t)n * 4, &pb, "sort permutation"));
  XL_TRY(dalloc(c, (size_t)n * 4, &ka, "sort keys"));
  XL_TRY(dalloc(c, (size_t)n * 4, &kb, "sort keys"));
  XL_TRY(dalloc(c, k::radix_temp_bytes(n), &tmp, "sort scratch"));
  HIP_TRY(c, k::iota_u32(pa.as<uint32_t>(), n, c->stream));
  for (int j = arity - 1; j >= 0; --j) {
    HIP_TRY(c, k::ordered_key(cols[j], types[j], pa.as<uint32_t>(), ka.as<uint32_t>(), n, c->stream));
    int alt = 0;
    HIP_TRY(c, k::radix_sort_u32(ka.as<uint32_t>(), pa.as<uint32_t>(), kb.as<uint32_t>(),
                                 pb.as<uint32_t>(), n, 32, tmp.p, c->stream, &alt));
    if (alt) std::swap(pa.p, pb.p);
  }
  std::swap(perm_out->p, pa.p);
  perm_out->c = c;
  return XL_OK;
}

xl_status compute_bounds(Context* c, Relation* r) {
  if (r->nrows == 0) return XL_OK;
  Buf mm;
  XL_TRY(dalloc(c, 8 * MAXC, &mm, "bounds"));
  int32_t init[2 * MAXC];
  for (int j = 0; j < MAXC; ++j) {
    init[2 * j] = INT32_MAX;
    init[2 * j + 1] = INT32_MIN;
  }
  HIP_TRY(c, hipMemcpyAsync(mm.p, init, sizeof(init), hipMemcpyHostToDevice, c->stream));
  for (int j = 0; j < r->arity; ++j)
    if (r->types[j] == T_I32)
      HIP_TRY(c, k::minmax_i32((const int32_t*)r->col[j], r->nrows, mm.as<int32_t>() + 2 * j, c->stream));
  int32_t out[2 * MAXC];
  XL_TRY(ctl_read(c, mm.p, sizeof(out), out));
  for (int j = 0; j < r->arity; ++j) {
    r->lo[j] = out[2 * j];
    r->hi[j] = out[2 * j + 1];
  }
  return XL_OK;
}

// Images of n order keys (device) of the 8-byte type lt: their ranks in the
// context's dictionary after the keys new to it are added.  Adding keys
// renumbers the dictionary, so every stored column of type lt is remapped
// (old rank -> new rank, order kept) and its relation gets a new generation.
xl_status dict_encode(Context* c, int lt, const u64* keys, int64_t n, uint32_t* images) {
  if (n <= 0) return XL_OK;
  const int64_t nd = c->dict_n[lt], nt = nd + n;
  Buf cat, alt, tmp, flag, pos, stmp, tot;
  XL_TRY(dalloc(c, (size_t)nt * 8, &cat, "dictionary merge"));
  XL_TRY(dalloc(c, (size_t)nt * 8, &alt, "dictionary merge"));
  XL_TRY(dalloc(c, k::radix_temp_bytes(nt), &tmp, "sort scratch"));
  if (nd > 0)
    HIP_TRY(c, hipMemcpyAsync(cat.p, c->dict[lt], (size_t)nd * 8, hipMemcpyDeviceToDevice, c->stream));
  HIP_TRY(c, hipMemcpyAsync(cat.as<u64>() + nd, keys, (size_t)n * 8, hipMemcpyDeviceToDevice, c->stream));
  int a = 0;
  HIP_TRY(c, k::radix_sort_u64(cat.as<u64>(), nullptr, alt.as<u64>(), nullptr, nt, 64, tmp.p, c->stream, &a));
  const u64* sorted = a ? alt.as<u64>() : cat.as<u64>();
  XL_TRY(dalloc(c, (size_t)nt * 4, &flag, "dictionary flags"));
  XL_TRY(dalloc(c, (size_t)nt * 4, &pos, "dictionary positions"));
  XL_TRY(dalloc(c, k::scan_temp_bytes(nt), &stmp, "scan scratch"));
  XL_TRY(dalloc(c, 8, &tot, "count"));
  HIP_TRY(c, k::unique_flags64(sorted, nt, flag.as<uint32_t>(), c->stream));
  HIP_TRY(c, k::scan_exclusive_u32(flag.as<uint32_t>(), pos.as<uint32_t>(), nt, tot.as<uint32_t>(), stmp.p,
                                   c->stream));
  uint32_t m = 0;
  XL_TRY(ctl_read(c, tot.p, 4, &m));
  if (m > (uint32_t)nd) {
    if (m >= (1u << 31))
      return c->fail(XL_CAPACITY_EXCEEDED, std::string("more than 2^31 distinct ") + type_name(lt) + " values");
    Buf nd_keys;
    XL_TRY(dalloc(c, (size_t)m * 8, &nd_keys, "type dictionary"));
    HIP_TRY(c, k::compact64(sorted, flag.as<uint32_t>(), pos.as<uint32_t>(), nd_keys.as<u64>(), nt, c->stream));
    if (nd > 0) {
      Buf map;
      XL_TRY(dalloc(c, (size_t)nd * 4, &map, "dictionary renumbering"));
      HIP_TRY(c, k::rank64(nd_keys.as<u64>(), m, c->dict[lt], nd, map.as<uint32_t>(), c->stream));
      for (Relation* r : c->rels) {
        bool touched = false;
        for (int j = 0; j < r->arity; ++j)
          if (r->ltypes[j] == lt && r->nrows > 0 && r->col[j]) {
            HIP_TRY(c, k::remap_codes(r->col[j], r->nrows, map.as<uint32_t>(), c->stream));
            touched = true;
          }
        if (touched) {
          r->generation = ++c->generations;
          c->icache_drop(r, true);
          XL_TRY(compute_bounds(c, r));
        }
      }
    }
    c->arena.release(c->dict[lt]);
    c->dict[lt] = (unsigned long long*)nd_keys.keep();
    c->dict_n[lt] = m;
  }
  HIP_TRY(c, k::rank64(c->dict[lt], c->dict_n[lt], keys, n, images, c->stream));
  return XL_OK;
}

// Int32 images of the columns of r given to a load (n values each, in host or
// device memory, packed at each type's element size) written to img[j] for
// the columns of type u32, bool, i64, u64 or f64.  The columns of one 8-byte
// type go through one dictionary update together, so no image of this load
// is renumbered by a later one.
xl_status encode_columns(Context* c, const Relation* r, const void* const* cols, int64_t n, int on_device,
                         uint32_t* const* img) {
  const hipMemcpyKind kind = on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
  for (int lt : {XL_U32, XL_BOOL}) {
    for (int j = 0; j < r->arity; ++j) {
      if (r->ltypes[j] != lt) continue;
      const size_t es = elem_bytes(lt);
      Buf in, bad;
      XL_TRY(dalloc(c, (size_t)n * es, &in, "loaded column"));
      XL_TRY(dalloc(c, 4, &bad, "check flag"));
      HIP_TRY(c, hipMemcpyAsync(in.p, cols[j], (size_t)n * es, kind, c->stream));
      HIP_TRY(c, hipMemsetAsync(bad.p, 0, 4, c->stream));
      HIP_TRY(c, k::encode_narrow(in.p, lt, n, img[j], bad.as<uint32_t>(), c->stream));
      uint32_t flag = 0;
      XL_TRY(ctl_read(c, bad.p, 4, &flag));
      if (flag)
        return c->fail(XL_INVALID_ARGUMENT,
                       "bool column " + std::to_string(j) + " of " + r->name + " holds a byte other than 0 or 1");
    }
  }
  for (int lt : {XL_I64, XL_U64, XL_F64}) {
    std::vector<int> js;
    for (int j = 0; j < r->arity; ++j)
      if (r->ltypes[j] == lt) js.push_back(j);
    if (js.empty()) continue;
    const int64_t m = n * (int64_t)js.size();
    Buf in, keys, imgs;
    XL_TRY(dalloc(c, (size_t)n * 8, &in, "loaded column"));
    XL_TRY(dalloc(c, (size_t)m * 8, &keys, "order keys"));
    XL_TRY(dalloc(c, (size_t)m * 4, &imgs, "column images"));
    for (size_t q = 0; q < js.size(); ++q) {
      HIP_TRY(c, hipMemcpyAsync(in.p, cols[js[q]], (size_t)n * 8, kind, c->stream));
      HIP_TRY(c, k::order_keys64(in.as<u64>(), lt, n, keys.as<u64>() + (int64_t)q * n, c->stream));
    }
    XL_TRY(dict_encode(c, lt, keys.as<u64>(), m, imgs.as<uint32_t>()));
    for (size_t q = 0; q < js.size(); ++q)
      HIP_TRY(c, hipMemcpyAsync(img[js[q]], imgs.as<uint32_t>() + (int64_t)q * n, (size_t)n * 4,
                                hipMemcpyDeviceToDevice, c->stream));
  }
  return XL_OK;
}

}  // namespace

// Give every constant of an 8-byte type in p's plans its current image,
// adding the values the dictionaries lack.
xl_status resolve_wide_constants(Program* p) {
  Context* c = p->ctx;
  for (int lt : {XL_I64, XL_U64, XL_F64}) {
    std::vector<u64> keys;
    std::vector<uint32_t*> dst;
    for (Stratum& st : p->strata)
      for (std::vector<RulePlan>* v : {&st.full, &st.variants})
        for (RulePlan& rp : *v)
          for (const WideConst& w : rp.wconsts) {
            if (w.ltype != lt) continue;
            keys.push_back(w.key);
            dst.push_back(w.where == 0   ? &rp.driver_act[w.a].cval
                          : w.where == 1 ? &rp.steps[w.a].act[w.b].cval
                                         : &rp.stage_consts[w.a][w.b]);
          }
    if (keys.empty()) continue;
    const int64_t n = (int64_t)keys.size();
    Buf dk, di;
    XL_TRY(dalloc(c, (size_t)n * 8, &dk, "constant keys"));
    XL_TRY(dalloc(c, (size_t)n * 4, &di, "constant images"));
    HIP_TRY(c, hipMemcpyAsync(dk.p, keys.data(), (size_t)n * 8, hipMemcpyHostToDevice, c->stream));
    XL_TRY(dict_encode(c, lt, dk.as<u64>(), n, di.as<uint32_t>()));
    std::vector<uint32_t> img((size_t)n);
    for (int64_t i0 = 0; i0 < n; i0 += 1024) {
      const int64_t m = std::min<int64_t>(1024, n - i0);
      XL_TRY(ctl_read(c, di.as<uint32_t>() + i0, (size_t)m * 4, img.data() + i0));
    }
    for (int64_t i = 0; i < n; ++i) *dst[(size_t)i] = img[(size_t)i];
  }
  return XL_OK;
}

// The gathered-round shape (see GatherShape).
bool gather_shape(const RulePlan& p, GatherShape* g) {
  if (!p.driver_delta || p.driver != p.head || p.driver->arity != 2 || p.steps.size() != 2 || p.nkey != 2 ||
      !p.negs.empty())
    return false;
  for (const auto& ops : p.stage_ops)
    if (!ops.empty()) return false;
  const ColAct &da = p.driver_act[0], &db = p.driver_act[1];
  if (da.kind != CA_BIND || db.kind != CA_BIND || da.slot == db.slot) return false;
  int ia = -1, ib = -1;
  for (int k = 0; k < 2; ++k) {
    if (p.steps[k].key_slot == da.slot) ia = k;
    else if (p.steps[k].key_slot == db.slot) ib = k;
  }
  if (ia < 0 || ib < 0) return false;
  auto other = [&](const StepPlan& st, int* col, int* slot) {
    if (st.rel == p.head || st.rel->arity != 2) return false;
    const int oc = 1 - st.key_col;
    if (st.act[oc].kind != CA_BIND) return false;
    *col = oc;
    *slot = st.act[oc].slot;
    return true;
  };
  int xs = -1, ys = -1;
  if (!other(p.steps[ia], &g->x_col, &xs) || !other(p.steps[ib], &g->y_col, &ys)) return false;
  if (xs != p.key_slot[0] || ys != p.key_slot[1] || xs == ys) return false;
  g->s1 = ia;
  g->s2 = ib;
  return true;
}

void relation_free_storage(Relation* r) {
  for (int j = 0; j < MAXC; ++j) {
    if (r->col[j]) r->ctx->arena.release(r->col[j]);
    r->col[j] = nullptr;
  }
  r->nrows = 0;
  r->sorted = false;
  r->generation = ++r->ctx->generations;  // cached indexes of the old rows no longer match
  r->ctx->icache_drop(r, true);
}

xl_status relation_clear(Relation* r) {
  relation_free_storage(r);
  return XL_OK;
}

// ================================================================== load / read
xl_status relation_load(Relation* r, const void* const* cols, int64_t n, int on_device) {
  Context* c = r->ctx;
  if (c->device < 0) return c->fail(XL_INVALID_ARGUMENT, "planning-only context cannot hold data");
  if (n < 0 || (n > 0 && !cols)) return c->fail(XL_INVALID_ARGUMENT, "bad row count or column pointers");
  if (n >= (int64_t)1 << 31) return c->fail(XL_CAPACITY_EXCEEDED, "relations hold fewer than 2^31 rows");
  for (int j = 0; j < r->arity && n > 0; ++j)
    if (!cols[j]) return c->fail(XL_INVALID_ARGUMENT, "null column pointer");
  if (n == 0) {
    relation_free_storage(r);
    return XL_OK;
  }
  Buf raw[MAXC];
  uint32_t* img[MAXC] = {};
  for (int j = 0; j < r->arity; ++j) {
    XL_TRY(dalloc(c, (size_t)n * 4, &raw[j], "loaded column"));
    img[j] = raw[j].as<uint32_t>();
    if (r->ltypes[j] == XL_I32 || r->ltypes[j] == XL_F32)
      HIP_TRY(c, hipMemcpyAsync(raw[j].p, cols[j], (size_t)n * 4,
                                on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice, c->stream));
  }
  XL_TRY(encode_columns(c, r, cols, n, on_device, img));
  int64_t m = n;
  Buf fin[MAXC];
  if (n == 1) {
    for (int j = 0; j < r->arity; ++j) std::swap(fin[j].p, raw[j].p), fin[j].c = c;
  } else {
    // sets: sort rows, flag rows that differ from their predecessor, compact
    uint32_t* rc[MAXC] = {};
    for (int j = 0; j < r->arity; ++j) rc[j] = raw[j].as<uint32_t>();
    Buf perm;
    XL_TRY(lex_perm(c, rc, r->types, r->arity, n, &perm));
    Buf sorted[MAXC];
    const uint32_t* sc[MAXC] = {};
    for (int j = 0; j < r->arity; ++j) {
      XL_TRY(dalloc(c, (size_t)n * 4, &sorted[j], "sorted column"));
      HIP_TRY(c, k::gather_u32(rc[j], perm.as<uint32_t>(), sorted[j].as<uint32_t>(), n, c->stream));
      sc[j] = sorted[j].as<uint32_t>();
      raw[j].reset();
    }
    Buf flag, pos, tmp, tot;
    XL_TRY(dalloc(c, (size_t)n * 4, &flag, "dedup flags"));
    XL_TRY(dalloc(c, (size_t)n * 4, &pos, "dedup positions"));
    XL_TRY(dalloc(c, k::scan_temp_bytes(n), &tmp, "scan scratch"));
    XL_TRY(dalloc(c, 8, &tot, "count"));
    HIP_TRY(c, k::row_change_flags(sc, r->arity, n, flag.as<uint32_t>(), c->stream));
    HIP_TRY(c, k::scan_exclusive_u32(flag.as<uint32_t>(), pos.as<uint32_t>(), n, tot.as<uint32_t>(),
                                     tmp.p, c->stream));
    uint32_t mm = 0;
    XL_TRY(ctl_read(c, tot.p, 4, &mm));
    m = mm;
    for (int j = 0; j < r->arity; ++j) {
      XL_TRY(dalloc(c, (size_t)m * 4, &fin[j], "relation column"));
      HIP_TRY(c, k::compact_u32(sc[j], flag.as<uint32_t>(), pos.as<uint32_t>(), fin[j].as<uint32_t>(),
                                n, c->stream));
    }
  }
  if (r->max_rows > 0 && m > r->max_rows)
    return c->fail(XL_CAPACITY_EXCEEDED, "relation " + r->name + " holds at most " +
                                             std::to_string(r->max_rows) + " rows, load has " +
                                             std::to_string(m));
  relation_free_storage(r);
  for (int j = 0; j < r->arity; ++j) r->col[j] = (uint32_t*)fin[j].keep();
  r->nrows = m;
  r->sorted = true;  // the deduplication above leaves the rows in lexicographic order
  XL_TRY(compute_bounds(c, r));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  return XL_OK;
}

xl_status relation_read(const Relation* r, void* const* cols, int64_t cap, int64_t* out_rows,
                        int on_device) {
  Context* c = r->ctx;
  if (cap < r->nrows) {
    if (out_rows) *out_rows = r->nrows;
    return c->fail(XL_CAPACITY_EXCEEDED, "output capacity " + std::to_string(cap) + " < " +
                                             std::to_string(r->nrows) + " rows of " + r->name);
  }
  const int64_t n = r->nrows;
  if (n > 0) {
    if (!cols) return c->fail(XL_INVALID_ARGUMENT, "null column pointers");
    for (int j = 0; j < r->arity; ++j)
      if (!cols[j]) return c->fail(XL_INVALID_ARGUMENT, "null column pointer");
    Buf perm;
    XL_TRY(lex_perm(c, r->col, r->types, r->arity, n, &perm));
    Buf stage, img;
    for (int j = 0; j < r->arity; ++j) {
      const int lt = r->ltypes[j];
      const size_t es = elem_bytes(lt);
      const bool plain = lt == XL_I32 || lt == XL_F32;
      // decode straight into the caller's device buffer when it is aligned
      // for the element size, else through device staging
      const bool direct = on_device && (uintptr_t)cols[j] % es == 0;
      if (!direct && !stage.p) XL_TRY(dalloc(c, (size_t)n * 8, &stage, "readout staging"));
      void* dst = direct ? cols[j] : stage.p;
      if (plain) {
        HIP_TRY(c, k::gather_u32(r->col[j], perm.as<uint32_t>(), (uint32_t*)dst, n, c->stream));
      } else {
        if (!img.p) XL_TRY(dalloc(c, (size_t)n * 4, &img, "readout images"));
        HIP_TRY(c, k::gather_u32(r->col[j], perm.as<uint32_t>(), img.as<uint32_t>(), n, c->stream));
        HIP_TRY(c, k::decode_column(img.as<uint32_t>(), n, lt, c->dict[lt], dst, c->stream));
      }
      if (!direct) {
        HIP_TRY(c, hipMemcpyAsync(cols[j], dst, (size_t)n * es, on_device ? hipMemcpyDeviceToDevice
                                                                           : hipMemcpyDeviceToHost, c->stream));
        HIP_TRY(c, hipStreamSynchronize(c->stream));
      }
    }
    HIP_TRY(c, hipStreamSynchronize(c->stream));
  }
  if (out_rows) *out_rows = n;
  return XL_OK;
}

// ================================================================== fixpoint run
namespace {

struct Interval {
  int64_t lo = INT64_MAX, hi = INT64_MIN;
  bool empty() const { return lo > hi; }
  void join(const Interval& o) {
    lo = std::min(lo, o.lo);
    hi = std::max(hi, o.hi);
  }
  static Interval full() { return {INT32_MIN, INT32_MAX}; }
};

struct DevIndex {
  Relation* rel = nullptr;
  int col = 0;
  int order_col = -1;  // >= 0: rows of one key ordered by this column (see order_kind)
  int order_kind = 0;  // 0: by the degree of the value, most first; 1: by the int32 value
  uint32_t* first = nullptr;  // with order_col: order_col value of each key's first row
  IndexProbe probe{};
  std::vector<std::unique_ptr<Buf>> owned;
};

// Sorted keys of a complete relation projected onto the columns a negated
// literal constrains.
struct DevNeg {
  Relation* rel = nullptr;
  int ncols = 0;
  int col[2] = {0, 0};
  Buf keys;
  int64_t n = 0;
};

struct HeadRun {
  Relation* rel = nullptr;
  Agg agg = Agg::NONE;
  int fold = k::FOLD_NONE;
  bool is_set = false, is_minmax = false, is_sortagg = false;
  int nkey = 1;
  KeyPack kp{};
  int bits0 = 1;      // width of the first packed key component
  double domain = 0;  // number of possible keys
  Buf table;
  int64_t cap = 0, keys = 0;
  // set heads: append-only row list of every tuple; the delta is a range
  Buf rows[2];
  int64_t rows_cap = 0, nrows = 0, dbeg = 0, dend = 0, round_begin = 0;
  int64_t round_new = 0;  // dense heads: tuples added this round
  // aggregate heads: delta rows (k0[, k1], value)
  Buf drow[3];
  int64_t dcap = 0, dn = 0;
  Buf didx;
  int64_t didx_n = 0;
  Buf ckey, cval;
  int64_t ccap = 0, cn = 0;
  uint32_t round = 0;
  int64_t preloaded = 0;
  // dense set heads: one bit per key of the (range0 x range1) key domain,
  // rows of row_bits bits indexed by the first key component
  bool dense = false;
  Buf bits;
  Buf dbits;  // tuples new in this round (same layout as bits)
  u64 row_bits = 0;
  uint32_t row_words = 0;
  int64_t range0 = 0;
  // frontier form (closure-shaped stratum over a dense two-column head): the
  // delta is one bitmap row per first-key value that gained tuples
  bool frontier = false;
  bool resident = false;        // frontier form run by one resident launch, which reads
                                // the seed's delta straight from dbits
  bool frontier_ready = false;  // the current delta is in fcnt/fdiff[fcur] (or dbits)
  Buf fx, fcnt[2], fdiff[2];    // delta row slot sg belongs to first-key value fx[sg]
  // gathered form (h(X,Y) :- e1(X,A), delta h(A,B), e2(Y,B)): the delta is
  // bitmap rows in dbits / gbits (by gcur) with one flag per row in gflag
  bool gathered = false;
  bool gather_ready = false;
  Buf gbits, gflag[2];
  Buf gbound[2];  // word bounds of the delta rows of dbits / gbits: lo[range0] then hi[range0]
  int gcur = 0;
  Buf hasin;                    // Y values with an in-edge (pull direction)
  int fcur = 0;
  int64_t fn = 0, fnew = 0;
  // dense count heads: one counter per key of the domain
  bool dcount = false;
  bool vbounds = false;  // the value column's bounds were read with the rows
  Buf counts;
  int64_t range1 = 1;
  // dense value heads (min/max): value array over (rank of the first key in
  // a dictionary of its possible values) x (second key - lo1), presence and
  // listed-this-round bits, and the dictionary (dmap: value - lo0 -> rank)
  bool dv = false;
  Buf dmap, dict, dvals, dpres, dchg;
  int64_t n0 = 0, dmap_n = 0;
  int64_t nrank_d = 0;  // sum/logsumexp heads: rank stride of the target-major delta slots (n0 rounded up to 32)
  std::vector<std::pair<Relation*, int>> dict_src;
  // dense sum/logsumexp heads (one carried-value variant): the same slots;
  // dvals/dpres hold the full relation, dcur/dcur_pres this round's delta,
  // dnext/dnext_pres the next one, dchg the keys marked for the pull
  bool ds = false;
  Buf dcur, dcur_pres, dnext, dnext_pres;
  Buf ndrow[3];
  bool pulled = false;
  int64_t pull_n = 0;
  // dense min/max heads with one carried-value variant: tiled rounds, the
  // delta rows grouped by rank (roff: first row of each rank)
  bool tiled = false;
  Buf roff;
  // e's rows grouped by (Z, tile of Y), built at the first tiled round
  std::vector<std::unique_ptr<Buf>> tcols;
  Buf toff;
  IndexProbe tidx{};
  uint32_t tile = 0, ntiles = 0;
  // key-column domains (bounds recorded on the materialized relation)
  int64_t dom_lo[2] = {0, 0}, dom_hi[2] = {0, 0};
  // batched rounds: this head's counters and round boundaries on the device
  // (row counts of its row list, or positions of the batch's slot list), the
  // base its emissions append at and its load limit
  u64* b_cnt = nullptr;
  u64* b_bnd = nullptr;
  u64 b_base = 0, b_limit = 0;
};

struct Runner {
  Context* c;
  Program* prog;
  xl_fixpoint_stats* st;
  std::vector<std::unique_ptr<DevIndex>> indexes;
  std::vector<std::unique_ptr<DevIndex>> kept;  // ready indexes made while materializing
  std::vector<std::unique_ptr<DevNeg>> negtabs;  // negation tables over complete relations
  std::vector<std::unique_ptr<HeadRun>> heads;
  int64_t cands = 0;
  hipEvent_t ev[2] = {nullptr, nullptr};
  ~Runner() {
    for (hipEvent_t e : ev)
      if (e) (void)hipEventDestroy(e);
  }

  // Slots of a dense value head's full relation and their layout (0: rank
  // major, n: target-major with n ranks per target, as sum/logsumexp heads).
  static int64_t full_slots(const HeadRun* h) {
    return h->ds ? h->nrank_d * h->range1 : std::max<int64_t>(h->n0, 1) * h->range1;
  }
  static uint32_t full_nrank(const HeadRun* h) { return h->ds ? (uint32_t)h->nrank_d : 0u; }

  HeadRun* head_of(const Relation* r) {
    for (auto& h : heads)
      if (h->rel == r) return h.get();
    return nullptr;
  }

  void record(int64_t rows) {
    if (st->rounds_recorded < XL_STATS_ROUNDS) st->delta_rows[st->rounds_recorded] = rows;
    st->rounds_recorded++;
  }

  // ------------------------------------------------------------ indexes
  // Index of rel by column col.  With order_col >= 0 the rows of each key are
  // further ordered: order_kind 0 by how many rows of rel have the order_col
  // value in column order_col (its out-degree when rel is an edge relation
  // indexed by its target), most first by base-8 class -- the
  // frontier pull scans in-edges
  // in that order, so that edges from well-connected sources, the likeliest
  // to be in a delta, come first; order_kind 1 by the int32 value itself
  // (the triangle join intersects sorted lists).
  // first (when given, with order_col >= 0) receives an array holding, per
  // key, the order_col value of the key's first row.
  xl_status get_index(Relation* rel, int col, IndexProbe* out, int order_col = -1,
                      const uint32_t** first = nullptr, int order_kind = 0, bool dense_only = false) {
    for (auto& ix : indexes)
      if (ix->rel == rel && ix->col == col && ix->order_col == order_col &&
          (order_col < 0 || ix->order_kind == order_kind) && (!dense_only || !ix->probe.keys)) {
        *out = ix->probe;
        if (first) *first = ix->first;
        return XL_OK;
      }
    const bool cacheable = c->index_cache_bytes > 0 && !head_of(rel);
    if (cacheable)
      for (CachedIndex& ce : c->icache)
        if (ce.rel == rel && ce.generation == rel->generation && ce.col == col && ce.order_col == order_col &&
            (!dense_only || !ce.probe.keys) &&
            (order_col < 0 || ce.order_kind == order_kind)) {
          ce.last_run = c->runs;
          auto ix = std::make_unique<DevIndex>();
          ix->rel = rel;
          ix->col = col;
          ix->order_col = order_col;
          ix->order_kind = order_kind;
          ix->probe = ce.probe;
          ix->first = ce.first;
          *out = ix->probe;
          if (first) *first = ix->first;
          indexes.push_back(std::move(ix));
          st->index_reuses++;
          return XL_OK;
        }
    st->index_builds++;
    auto ix = std::make_unique<DevIndex>();
    ix->rel = rel;
    ix->col = col;
    ix->order_col = order_col;
    ix->order_kind = order_kind;
    IndexProbe& p = ix->probe;
    p.ncols = rel->arity;
    auto own = [&](size_t bytes, const char* what, void** ptr) -> xl_status {
      ix->owned.push_back(std::make_unique<Buf>());
      XL_TRY(dalloc(c, bytes, ix->owned.back().get(), what));
      *ptr = ix->owned.back()->p;
      return XL_OK;
    };
    // rows as this round sees them: a head of the running stratum (a
    // self-join) contributes its current full relation
    const uint32_t* rcol[MAXC] = {};
    int64_t n = rel->nrows;
    int32_t klo = rel->lo[col], khi = rel->hi[col];
    for (int j = 0; j < rel->arity; ++j) rcol[j] = rel->col[j];
    if (HeadRun* h = head_of(rel)) {
      if (h->frontier || h->dcount || h->is_sortagg || col >= h->nkey)
        return c->fail(XL_UNSUPPORTED, "relation " + rel->name + " cannot be joined inside its own stratum");
      klo = (int32_t)h->dom_lo[col];
      khi = (int32_t)h->dom_hi[col];
      if (h->dense) {  // rows of the current bitmap, in key order
        n = h->keys;
        void* snap[2] = {nullptr, nullptr};
        for (int j = 0; j < h->nkey; ++j) XL_TRY(own((size_t)std::max<int64_t>(n, 1) * 4, "head snapshot", &snap[j]));
        Buf tmp, tot;
        if (h->nkey == 2) {
          Buf cnt, off;
          XL_TRY(dalloc(c, (size_t)h->range0 * 4, &cnt, "row counts"));
          XL_TRY(dalloc(c, (size_t)(h->range0 + 1) * 4, &off, "row offsets"));
          XL_TRY(dalloc(c, k::scan_temp_bytes(h->range0), &tmp, "scan scratch"));
          HIP_TRY(c, k::row_popcount(h->bits.as<uint32_t>(), h->range0, h->row_words, cnt.as<uint32_t>(), c->stream));
          HIP_TRY(c, k::scan_exclusive_u32(cnt.as<uint32_t>(), off.as<uint32_t>(), h->range0,
                                           off.as<uint32_t>() + h->range0, tmp.p, c->stream));
          HIP_TRY(c, k::bits_to_rows(h->bits.as<uint32_t>(), h->range0, h->row_words, off.as<uint32_t>(),
                                     h->kp.lo[0], h->kp.lo[1], (uint32_t*)snap[0], (uint32_t*)snap[1], n,
                                     c->stream));
          HIP_TRY(c, k::check_eq(off.as<uint32_t>() + h->range0, (uint32_t)n, c->dcheck, CHECK_BITMAP_ROWS,
                                 c->stream));
        } else {
          const int64_t nbits = (h->range0 + 31) / 32 * 32;
          XL_TRY(dalloc(c, k::bits_list_temp_bytes(nbits), &tmp, "compaction scratch"));
          XL_TRY(dalloc(c, 8, &tot, "count"));
          for (int pass = 0; pass < 2; ++pass)
            HIP_TRY(c, k::bits_keys(h->bits.as<uint32_t>(), nbits, 1, h->kp.lo[0], 0, 1, false, (uint32_t*)snap[0],
                                    nullptr, tot.as<uint32_t>(), tmp.p, pass == 1, c->stream));
        }
        for (int j = 0; j < h->nkey; ++j) rcol[j] = (const uint32_t*)snap[j];
      } else if (h->is_set) {
        n = h->nrows;
        for (int j = 0; j < h->nkey; ++j) rcol[j] = h->rows[j].as<uint32_t>();
      } else {  // min/max: compact a snapshot of the current keys and values
        n = h->keys;
        void* snap[3];
        for (int j = 0; j <= h->nkey; ++j) XL_TRY(own((size_t)std::max<int64_t>(n, 1) * 4, "head snapshot", &snap[j]));
        Buf tmp, tot;
        const int64_t ns = h->dv ? full_slots(h) : h->cap;
        XL_TRY(dalloc(c, k::compact_temp_bytes(ns), &tmp, "compaction scratch"));
        XL_TRY(dalloc(c, 8, &tot, "count"));
        uint32_t* k1 = h->nkey == 2 ? (uint32_t*)snap[1] : nullptr;
        if (h->dv)
          HIP_TRY(c, k::dense_rows(h->dvals.as<uint32_t>(), h->dpres.as<uint32_t>(), h->dict.as<uint32_t>(), ns,
                                   h->range1, full_nrank(h), h->kp, rel->types[h->nkey], h->fold, (uint32_t*)snap[0], k1,
                                   (uint32_t*)snap[h->nkey], std::max<int64_t>(n, 1), tot.as<uint32_t>(), tmp.p,
                                   c->stream));
        else
          HIP_TRY(c, k::table16_compact(h->table.as<Slot16>(), h->cap, h->kp, rel->types[h->nkey], h->fold,
                                        (uint32_t*)snap[0], k1, (uint32_t*)snap[h->nkey], std::max<int64_t>(n, 1),
                                        tot.as<uint32_t>(), tmp.p, c->stream));
        for (int j = 0; j <= h->nkey; ++j) rcol[j] = (const uint32_t*)snap[j];
      }
    }
    if (n == 0) {
      void* off;
      XL_TRY(own(8, "index offsets", &off));
      HIP_TRY(c, hipMemsetAsync(off, 0, 8, c->stream));
      p.off = (uint32_t*)off;
      p.keys = nullptr;
      p.key_lo = 0;
      p.key_range = 0;
    } else {
      if (rel->types[col] != T_I32) return c->fail(XL_UNSUPPORTED, "index key columns must be int32");
      const int64_t range = (int64_t)khi - klo + 1;
      const bool ordered = order_col >= 0 && order_col < rel->arity && rel->types[order_col] == T_I32;
      // Direct-address offsets over a dense key range; a compacted index
      // (distinct keys, found by binary search) over a wide or sparse one.
      // The kernels that address per-key arrays by key value (frontier,
      // tiled, pull and gathered rounds, index degrees, degree order) ask for
      // the direct form; it and ordered indexes keep at most 2^25 rows.
      const bool compact = !dense_only && (order_col < 0 || order_kind == 1) &&
                           (range > ((int64_t)1 << 30) || (range > ((int64_t)1 << 22) && range > 16 * n));
      if ((dense_only || ordered) && n > ((int64_t)1 << 25))
        return c->fail(XL_UNSUPPORTED, "indexed relation " + rel->name + " exceeds 2^25 rows for this join form");
      if (!compact && range > ((int64_t)1 << 30))
        return c->fail(XL_UNSUPPORTED, "key range of " + rel->name + " column " + std::to_string(col) +
                                           " exceeds 2^30 values for this join form");
      const int kbits = std::max(1, bitlen((uint64_t)range - 1));
      // offsets from ascending key images: direct over the range, or compacted
      auto offsets = [&](const uint32_t* sorted_keys) -> xl_status {
        void* off;
        if (!compact) {
          XL_TRY(own((size_t)(range + 1) * 4, "index offsets", &off));
          HIP_TRY(c, k::csr_offsets(sorted_keys, n, (uint32_t)range, (uint32_t*)off, c->stream));
          p.off = (uint32_t*)off;
          p.keys = nullptr;
          p.key_range = (uint32_t)range;
          return XL_OK;
        }
        void* uk;
        Buf tmp, cnt;
        XL_TRY(own((size_t)(n + 1) * 4, "index offsets", &off));
        XL_TRY(own((size_t)n * 4, "index keys", &uk));
        XL_TRY(dalloc(c, k::compact_offsets_temp_bytes(n), &tmp, "index compaction scratch"));
        XL_TRY(dalloc(c, 8, &cnt, "count"));
        HIP_TRY(c, k::compact_offsets(sorted_keys, n, (uint32_t*)uk, (uint32_t*)off, cnt.as<uint32_t>(), tmp.p,
                                      c->stream));
        uint32_t nk = 0;
        XL_TRY(ctl_read(c, cnt.p, 4, &nk));
        p.off = (uint32_t*)off;
        p.keys = (const uint32_t*)uk;
        p.key_range = nk;
        return XL_OK;
      };
      // A loaded relation keeps its rows in lexicographic order, so its index
      // by the first column -- plain, or ordered by the second column's
      // values -- is its rows as they are: only the offsets are built, and
      // the index reads the relation's own columns.
      const bool presorted = !head_of(rel) && rel->sorted && col == 0 &&
                             (order_col < 0 || (ordered && order_col == 1 && order_kind == 1));
      if (presorted) {
        Buf keys;
        XL_TRY(dalloc(c, (size_t)n * 4, &keys, "index keys"));
        HIP_TRY(c, k::sub_lo(rcol[col], klo, keys.as<uint32_t>(), n, c->stream));
        XL_TRY(offsets(keys.as<uint32_t>()));
        for (int j = 0; j < rel->arity; ++j) p.col[j] = rcol[j];
        p.key_lo = klo;
        *out = p;
        if (first) *first = ix->first;
        if (cacheable) cache_index(*ix);
        indexes.push_back(std::move(ix));
        return XL_OK;
      }
      Buf perm, perm2, tmp;
      XL_TRY(dalloc(c, (size_t)n * 4, &perm, "index permutation"));
      XL_TRY(dalloc(c, (size_t)n * 4, &perm2, "index permutation"));
      XL_TRY(dalloc(c, k::radix_temp_bytes(n), &tmp, "sort scratch"));
      uint32_t* sp = nullptr;
      if (ordered) {
        // one sort by (key, order value), of 32-bit composite keys when
        // both parts fit; the offsets come from the sorted keys' high bits.
        // Degree order reads each order value's degree from the plain
        // index of rel by the order column (its row count as a key there).
        IndexProbe dz{};
        if (order_kind == 0) XL_TRY(get_index(rel, order_col, &dz, -1, nullptr, 0, true));
        // value order: the order column's bounds when known (a finished
        // relation, or a key column of a head), else the whole int32 range
        int32_t vlo = INT32_MIN;
        int vbits = 32;
        if (order_kind == 1) {
          HeadRun* oh = head_of(rel);
          if (!oh && rel->nrows > 0) {
            vlo = rel->lo[order_col];
            vbits = std::max(1, bitlen((uint64_t)((int64_t)rel->hi[order_col] - rel->lo[order_col])));
          } else if (oh && order_col < oh->nkey) {
            vlo = (int32_t)oh->dom_lo[order_col];
            vbits = std::max(1, bitlen((uint64_t)(oh->dom_hi[order_col] - oh->dom_lo[order_col])));
          }
        }
        const int obits = order_kind == 1 ? vbits : 2;  // degree order: four base-8 classes
        const bool wide = obits + kbits > 32;
        const size_t kw = wide ? 8 : 4;
        Buf ka, kb;
        XL_TRY(dalloc(c, (size_t)n * kw, &ka, "index order keys"));
        XL_TRY(dalloc(c, (size_t)n * kw, &kb, "index order keys"));
        HIP_TRY(c, k::order_keys(rcol[col], klo, rcol[order_col], order_kind == 1 ? vlo : dz.key_lo, obits,
                                 order_kind == 1 ? nullptr : dz.off, dz.key_range, n, ka.p, wide,
                                 perm.as<uint32_t>(), c->stream));
        int alt = 0;
        if (wide)
          HIP_TRY(c, k::radix_sort_u64(ka.as<u64>(), perm.as<uint32_t>(), kb.as<u64>(), perm2.as<uint32_t>(), n,
                                       obits + kbits, tmp.p, c->stream, &alt));
        else
          HIP_TRY(c, k::radix_sort_u32(ka.as<uint32_t>(), perm.as<uint32_t>(), kb.as<uint32_t>(),
                                       perm2.as<uint32_t>(), n, obits + kbits, tmp.p, c->stream, &alt));
        sp = alt ? perm2.as<uint32_t>() : perm.as<uint32_t>();
        const void* sk = alt ? kb.p : ka.p;
        if (!compact) {
          void* off;
          XL_TRY(own((size_t)(range + 1) * 4, "index offsets", &off));
          HIP_TRY(c, k::csr_offsets_high(sk, wide, obits, n, (uint32_t)range, (uint32_t*)off, c->stream));
          p.off = (uint32_t*)off;
          p.keys = nullptr;
          p.key_range = (uint32_t)range;
        } else {
          Buf keys;
          XL_TRY(dalloc(c, (size_t)n * 4, &keys, "index keys"));
          HIP_TRY(c, k::high_bits(sk, wide, obits, n, keys.as<uint32_t>(), c->stream));
          XL_TRY(offsets(keys.as<uint32_t>()));
        }
      } else {
        Buf keys, keys2;
        XL_TRY(dalloc(c, (size_t)n * 4, &keys, "index keys"));
        XL_TRY(dalloc(c, (size_t)n * 4, &keys2, "index keys"));
        HIP_TRY(c, k::keys_perm(rcol[col], klo, n, keys.as<uint32_t>(), perm.as<uint32_t>(), c->stream));
        int alt = 0;
        HIP_TRY(c, k::radix_sort_u32(keys.as<uint32_t>(), perm.as<uint32_t>(), keys2.as<uint32_t>(),
                                     perm2.as<uint32_t>(), n, kbits, tmp.p, c->stream, &alt));
        const uint32_t* sk = alt ? keys2.as<uint32_t>() : keys.as<uint32_t>();
        sp = alt ? perm2.as<uint32_t>() : perm.as<uint32_t>();
        XL_TRY(offsets(sk));
      }
      uint32_t* cols[MAXC] = {};
      for (int j = 0; j < rel->arity; ++j) {
        void* cj;
        XL_TRY(own((size_t)n * 4, "index column", &cj));
        cols[j] = (uint32_t*)cj;
        p.col[j] = cols[j];
      }
      HIP_TRY(c, k::gather_cols(rcol, cols, rel->arity, sp, n, c->stream));
      if (ordered && order_kind == 0) {
        void* fp;
        XL_TRY(own((size_t)range * 4, "index first rows", &fp));
        HIP_TRY(c, k::segment_first(p.off, p.col[order_col], (uint32_t)range, (uint32_t*)fp, c->stream));
        ix->first = (uint32_t*)fp;
      }
      p.key_lo = klo;
    }
    *out = p;
    if (first) *first = ix->first;
    if (cacheable) cache_index(*ix);
    indexes.push_back(std::move(ix));
    return XL_OK;
  }

  // Hand a freshly built index of a relation that is not a head to the
  // context's cache (its blocks then outlive the run), and evict the least
  // recently used entries not used by this run while the cache is over its
  // budget.
  void cache_index(DevIndex& ix) {
    CachedIndex ce;
    ce.rel = ix.rel;
    ce.generation = ix.rel->generation;
    ce.col = ix.col;
    ce.order_col = ix.order_col;
    ce.order_kind = ix.order_kind;
    ce.probe = ix.probe;
    ce.first = ix.first;
    ce.last_run = c->runs;
    for (auto& b : ix.owned) {
      ce.bytes += c->arena.block_size(b->p);
      ce.blocks.push_back(b->keep());
    }
    ix.owned.clear();
    c->icache.push_back(std::move(ce));
    size_t total = 0;
    for (const CachedIndex& e : c->icache) total += e.bytes;
    while (total > c->index_cache_bytes) {
      int victim = -1;
      for (int i = 0; i < (int)c->icache.size(); ++i)
        if (c->icache[i].last_run != c->runs &&
            (victim < 0 || c->icache[i].last_run < c->icache[victim].last_run))
          victim = i;
      if (victim < 0) break;  // every entry serves the running program
      total -= c->icache[victim].bytes;
      for (void* b : c->icache[victim].blocks) c->arena.release(b);
      c->icache.erase(c->icache.begin() + victim);
    }
  }

  // ------------------------------------------------------------ domains / heads
  Interval col_interval(Relation* rel, int col, const std::map<Relation*, std::vector<Interval>>& dom) {
    auto it = dom.find(rel);
    if (it != dom.end()) {
      if (col < (int)it->second.size()) return it->second[col];
      return Interval::full();
    }
    if (rel->nrows == 0) return Interval{};
    if (rel->types[col] != T_I32) return Interval::full();
    return Interval{rel->lo[col], rel->hi[col]};
  }

  // A min/max head can use a dense value array when every rule binds its
  // first key from a finished relation's column (a superset of the values it
  // can take) or carries it over from the head's own first column.  The
  // dictionary is the union of those columns (and of rows already loaded
  // into the head).
  void plan_dense_values(const Stratum& s, HeadRun* hr) {
    Relation* h = hr->rel;
    const int64_t r0 = hr->dom_hi[0] - hr->dom_lo[0] + 1;
    const int64_t r1 = hr->nkey == 2 ? hr->dom_hi[1] - hr->dom_lo[1] + 1 : 1;
    if (r0 <= 0 || r0 > ((int64_t)1 << 28) || r1 <= 0 || r1 > ((int64_t)1 << 30)) return;
    // the dictionary build needs two arrays over the first key's range, and
    // the arrays one row per dictionary value over the second key's range:
    // with the budget init_dv applies to the arrays, skip the dense form
    // before building a dictionary that could not be used
    const double budget = std::min(8589934592.0, (double)c->arena.capacity() / 4);
    if ((double)r0 * 8 > budget || (double)r1 * 16.5 > budget) return;
    std::vector<std::pair<Relation*, int>> src;
    for (const RulePlan& p : s.full) {
      if (p.head != h) continue;
      const int sl = p.key_slot[0];
      if (p.var_is_arith[sl]) return;
      bool carried = false;
      std::pair<Relation*, int> best{nullptr, 0};
      for (const auto& vs : p.var_sources[sl]) {
        if (vs.first == h && vs.second == 0) carried = true;
        bool in_stratum = false;
        for (Relation* o : s.heads) in_stratum = in_stratum || o == vs.first;
        if (in_stratum || vs.first->types[vs.second] != T_I32) continue;
        if (!best.first || vs.first->nrows < best.first->nrows) best = vs;
      }
      if (carried) continue;
      if (!best.first) return;
      src.push_back(best);
    }
    if (hr->is_minmax && h->nrows > 0) src.push_back({h, 0});  // loaded rows
    hr->dv = true;
    hr->dmap_n = r0;
    hr->range1 = (r1 + 31) / 32 * 32;  // rank rows start on word boundaries
    hr->dict_src = src;
  }

  xl_status setup_heads(Stratum& s) {
    std::map<Relation*, std::vector<Interval>> dom;
    for (Relation* h : s.heads) {
      const Agg a = prog->head_agg(h);
      const int nkey = h->arity - (a != Agg::NONE ? 1 : 0);
      std::vector<Interval> d(nkey);
      const bool keep = a == Agg::NONE || a == Agg::MIN || a == Agg::MAX;
      if (keep && h->nrows > 0)
        for (int j = 0; j < nkey; ++j) d[j] = Interval{h->lo[j], h->hi[j]};
      dom[h] = d;
    }
    for (int iter = 0; iter < 64; ++iter) {
      bool changed = false;
      for (RulePlan& p : s.full) {
        std::vector<Interval>& d = dom[p.head];
        for (int j = 0; j < p.nkey; ++j) {
          const int sl = p.key_slot[j];
          Interval iv;
          if (p.var_is_arith[sl]) {
            iv = Interval::full();
          } else {
            iv = Interval::full();
            for (auto& src : p.var_sources[sl]) {
              Interval o = col_interval(src.first, src.second, dom);
              iv.lo = std::max(iv.lo, o.lo);
              iv.hi = std::min(iv.hi, o.hi);
            }
          }
          if (iv.empty()) continue;
          Interval before = d[j];
          d[j].join(iv);
          changed = changed || before.lo != d[j].lo || before.hi != d[j].hi;
        }
      }
      if (!changed) break;
    }
    for (Relation* h : s.heads) {
      auto hr = std::make_unique<HeadRun>();
      hr->rel = h;
      hr->agg = prog->head_agg(h);
      hr->nkey = h->arity - (hr->agg != Agg::NONE ? 1 : 0);
      hr->is_set = hr->agg == Agg::NONE;
      hr->is_minmax = hr->agg == Agg::MIN || hr->agg == Agg::MAX;
      hr->is_sortagg = !hr->is_set && !hr->is_minmax;
      switch (hr->agg) {
        case Agg::COUNT: hr->fold = k::FOLD_COUNT; break;
        case Agg::SUM: hr->fold = k::FOLD_SUM; break;
        case Agg::MIN: hr->fold = k::FOLD_MIN; break;
        case Agg::MAX: hr->fold = k::FOLD_MAX; break;
        case Agg::LSE: hr->fold = k::FOLD_LSE; break;
        default: hr->fold = k::FOLD_NONE;
      }
      std::vector<Interval>& d = dom[h];
      KeyPack kp{};
      kp.nkey = hr->nkey;
      int bits0 = 1;
      double dsize = 1;
      int full = 0;  // key columns whose domain spans all 2^32 values
      for (int j = 0; j < hr->nkey; ++j) {
        Interval iv = d[j].empty() ? Interval{0, 0} : d[j];
        kp.lo[j] = (int32_t)iv.lo;
        const int b = std::max(1, bitlen((uint64_t)(iv.hi - iv.lo)));
        if (j == 0) bits0 = b; else kp.shift = b;
        dsize *= (double)(iv.hi - iv.lo + 1);
        full += iv.hi - iv.lo == 0xffffffffll;
      }
      // a packed key is all ones (the empty-slot marker of the hash tables)
      // only for the largest tuple of two key domains of 2^32 values each
      if (hr->nkey == 2 && full == 2)
        return c->fail(XL_UNSUPPORTED, "both key columns of " + h->name + " span all 2^32 values");
      hr->kp = kp;
      hr->bits0 = bits0;
      hr->domain = dsize;
      for (int j = 0; j < hr->nkey; ++j) {
        const Interval iv = d[j].empty() ? Interval{0, 0} : d[j];
        hr->dom_lo[j] = iv.lo;
        hr->dom_hi[j] = iv.hi;
      }
      if (hr->agg == Agg::COUNT && c->index_mode != 1) {
        const int64_t r0 = hr->dom_hi[0] - hr->dom_lo[0] + 1;
        const int64_t r1 = hr->nkey == 2 ? hr->dom_hi[1] - hr->dom_lo[1] + 1 : 1;
        if ((double)r0 * (double)r1 * 4 <= std::min(4294967296.0, (double)c->arena.capacity() / 8)) {
          hr->dcount = true;
          hr->range0 = r0;
          hr->range1 = r1;
        }
      }
      if (hr->is_minmax && c->index_mode != 1) {
        plan_dense_values(s, hr.get());
        hr->tiled = hr->dv && hr->nkey == 2 && c->dense_tiles >= 0 && s.recursive && s.heads.size() == 1 &&
                    s.variants.size() == 1 && s.variants[0].carried_val;
      }
      if ((hr->agg == Agg::SUM || hr->agg == Agg::LSE) && hr->nkey == 2 && c->index_mode != 1 && s.recursive &&
          s.heads.size() == 1 && s.variants.size() == 1 && s.variants[0].carried_val) {
        plan_dense_values(s, hr.get());
        hr->ds = hr->dv;
      }
      if (hr->is_set && c->index_mode != 1) {
        const Interval i0 = d[0].empty() ? Interval{0, 0} : d[0];
        const int64_t range0 = i0.hi - i0.lo + 1;
        int64_t range1 = 1;
        if (hr->nkey == 2) {
          const Interval i1 = d[1].empty() ? Interval{0, 0} : d[1];
          range1 = i1.hi - i1.lo + 1;
        }
        const u64 row_bits = hr->nkey == 2 ? (u64)((range1 + 31) / 32) * 32 : 1;
        const double total_bits = hr->nkey == 2 ? (double)range0 * (double)row_bits
                                                : (double)((range0 + 31) / 32) * 32.0;
        const double budget = c->index_mode == 2 ? (double)c->arena.capacity() / 2
                                                 : std::min(4294967296.0, (double)c->arena.capacity() / 4);
        if (total_bits / 8 <= budget) {
          hr->dense = true;
          hr->range0 = range0;
          hr->row_bits = row_bits;
          hr->row_words = (uint32_t)std::min<u64>(row_bits / 32, 0xffffffffull);
          // frontier form: the stratum is this head alone with one closure-shaped
          // variant; its kernel stages three rows of row_words words plus about
          // 19 KB in LDS, which must stay within a workgroup's 64 KB
          hr->frontier = s.recursive && s.heads.size() == 1 && s.variants.size() == 1 &&
                         s.variants[0].carried && hr->nkey == 2 && hr->row_words <= 3072 &&
                         total_bits / 8 * 3 <= budget;
          hr->resident = hr->frontier && c->frontier_resident;
          GatherShape gs;
          hr->gathered = !hr->frontier && c->gather_rounds && s.recursive && s.heads.size() == 1 &&
                         s.variants.size() == 1 && hr->nkey == 2 && hr->is_set && hr->row_words <= 3072 &&
                         total_bits / 8 * 2 <= budget && gather_shape(s.variants[0], &gs);
        }
      }
      hr->preloaded = (hr->is_set || hr->is_minmax) ? h->nrows : 0;
      XL_TRY(init_head(hr.get()));
      heads.push_back(std::move(hr));
    }
    return XL_OK;
  }

  size_t slot_bytes(const HeadRun* h) const { return h->is_set ? 8 : sizeof(Slot16); }

  xl_status alloc_table(HeadRun* h, int64_t cap, Buf* out) {
    XL_TRY(dalloc(c, (size_t)cap * slot_bytes(h), out, "hash table"));
    HIP_TRY(c, k::fill_bytes(out->p, 0xff, (size_t)cap * slot_bytes(h), c->stream));
    return XL_OK;
  }

  int64_t initial_cap(int64_t expect) {
    int64_t cap = (int64_t)1 << c->hash_min_log2;
    return (int64_t)std::max<uint64_t>(cap, next_pow2((uint64_t)std::max<int64_t>(expect, 1) * 4));
  }

  xl_status init_dense(HeadRun* h) {
    Relation* r = h->rel;
    const double total_bits = h->nkey == 2 ? (double)h->range0 * (double)h->row_bits
                                           : (double)((h->range0 + 31) / 32) * 32.0;
    const size_t bytes = (size_t)(total_bits / 8);
    XL_TRY(dalloc(c, bytes, &h->bits, "dense key bitmap"));
    HIP_TRY(c, k::fill_bytes(h->bits.p, 0, bytes, c->stream));
    XL_TRY(dalloc(c, bytes, &h->dbits, "dense delta bitmap"));
    HIP_TRY(c, k::fill_bytes(h->dbits.p, 0, bytes, c->stream));
    // the row list only holds loaded rows (the seed scans them); derived
    // tuples live in the bitmap and each round's delta in dbits
    h->rows_cap = std::max<int64_t>(h->preloaded, 1);
    for (int j = 0; j < h->nkey; ++j) {
      XL_TRY(dalloc(c, (size_t)h->rows_cap * 4, &h->rows[j], "relation rows"));
      if (h->preloaded)
        HIP_TRY(c, hipMemcpyAsync(h->rows[j].p, r->col[j], (size_t)h->preloaded * 4,
                                  hipMemcpyDeviceToDevice, c->stream));
    }
    HIP_TRY(c, k::bits_set_rows(h->bits.as<uint32_t>(), h->row_bits, h->rows[0].as<uint32_t>(),
                                h->nkey == 2 ? h->rows[1].as<uint32_t>() : nullptr, h->preloaded, h->kp,
                                c->stream));
    h->nrows = h->keys = h->preloaded;
    h->dbeg = h->dend = 0;
    if (h->gathered) {
      XL_TRY(dalloc(c, bytes, &h->gbits, "dense delta bitmap"));
      HIP_TRY(c, k::fill_bytes(h->gbits.p, 0, bytes, c->stream));
      for (int b = 0; b < 2; ++b) {
        XL_TRY(dalloc(c, (size_t)std::max<int64_t>(h->range0, 1) * 4, &h->gflag[b], "delta row flags"));
        HIP_TRY(c, hipMemsetAsync(h->gflag[b].p, 0, (size_t)std::max<int64_t>(h->range0, 1) * 4, c->stream));
        XL_TRY(dalloc(c, (size_t)std::max<int64_t>(h->range0, 1) * 8, &h->gbound[b], "delta row bounds"));
        HIP_TRY(c, k::fill_bounds(h->gbound[b].as<uint32_t>(), h->gbound[b].as<uint32_t>() + h->range0, h->range0,
                                  (uint32_t)h->row_words, 0u, c->stream));
      }
    }
    if (h->frontier && !h->resident) {
      XL_TRY(dalloc(c, (size_t)std::max<int64_t>(h->range0, 1) * 4, &h->fx, "delta row keys"));
      for (int b = 0; b < 2; ++b) {
        XL_TRY(dalloc(c, (size_t)std::max<int64_t>(h->range0, 1) * 4, &h->fcnt[b], "delta row counts"));
        XL_TRY(dalloc(c, (size_t)std::max<int64_t>(h->range0, 1) * h->row_words * 4, &h->fdiff[b],
                      "delta bitmap rows"));
      }
    }
    return XL_OK;
  }

  xl_status init_dcount(HeadRun* h) {
    const size_t bytes = (size_t)h->range0 * (size_t)h->range1 * 4;
    XL_TRY(dalloc(c, bytes, &h->counts, "dense counters"));
    HIP_TRY(c, k::fill_bytes(h->counts.p, 0, bytes, c->stream));
    return XL_OK;
  }



  // Build the first-key dictionary, then the dense arrays if they fit; a
  // head that does not fit falls back to the hash table (h->dv cleared).
  xl_status init_dv(HeadRun* h) {
    Relation* r = h->rel;
    const uint32_t range = (uint32_t)h->dmap_n;
    Buf pos, tmp, tot;
    XL_TRY(dalloc(c, (size_t)range * 4, &h->dmap, "key dictionary map"));
    HIP_TRY(c, hipMemsetAsync(h->dmap.p, 0, (size_t)range * 4, c->stream));
    for (const auto& sc : h->dict_src) {
      const int64_t n = sc.first == r ? h->preloaded : sc.first->nrows;
      HIP_TRY(c, k::dict_mark(sc.first->col[sc.second], n, h->kp.lo[0], range, h->dmap.as<uint32_t>(),
                              c->stream));
    }
    XL_TRY(dalloc(c, (size_t)range * 4, &pos, "key dictionary ranks"));
    XL_TRY(dalloc(c, k::scan_temp_bytes(range), &tmp, "scan scratch"));
    XL_TRY(dalloc(c, 8, &tot, "count"));
    HIP_TRY(c, k::scan_exclusive_u32(h->dmap.as<uint32_t>(), pos.as<uint32_t>(), range, tot.as<uint32_t>(),
                                     tmp.p, c->stream));
    uint32_t n0 = 0;
    XL_TRY(ctl_read(c, tot.p, 4, &n0));
    h->n0 = n0;
    const double slots = (double)std::max<uint32_t>(n0, 1) * (double)h->range1;
    // sum/logsumexp heads pad the ranks to whole words: their slot indices
    // (32-bit in the kernels) run up to the padded count
    const double padded = h->ds ? (double)((std::max<uint32_t>(n0, 1) + 31) / 32 * 32) * (double)h->range1 : slots;
    const double budget = std::min(8589934592.0, (double)c->arena.capacity() / 4);
    if (padded >= 4294967296.0 || padded * (h->ds ? 16.5 : 8.25) > budget) {
      h->dv = h->ds = h->tiled = false;
      h->dmap.reset();
      return XL_OK;
    }
    XL_TRY(dalloc(c, (size_t)std::max<uint32_t>(n0, 1) * 4, &h->dict, "key dictionary"));
    HIP_TRY(c, k::dict_finish(h->dmap.as<uint32_t>(), pos.as<uint32_t>(), range, h->kp.lo[0],
                              h->dict.as<uint32_t>(), c->stream));
    // sum/logsumexp heads lay the full relation out like their delta slots
    // (target-major, ranks padded to whole words)
    if (h->ds) h->nrank_d = (std::max<int64_t>(n0, 1) + 31) / 32 * 32;
    const size_t ns = h->ds ? (size_t)h->nrank_d * (size_t)h->range1 : (size_t)slots, nw = (ns + 31) / 32;
    XL_TRY(dalloc(c, ns * 4, &h->dvals, "dense values"));
    XL_TRY(dalloc(c, nw * 4, &h->dpres, "dense presence bits"));
    XL_TRY(dalloc(c, nw * 4, &h->dchg, "dense delta bits"));
    HIP_TRY(c, k::fill_bytes(h->dvals.p, 0xff, ns * 4, c->stream));
    HIP_TRY(c, k::fill_bytes(h->dpres.p, 0, nw * 4, c->stream));
    HIP_TRY(c, k::fill_bytes(h->dchg.p, 0, nw * 4, c->stream));
    if (h->tiled) XL_TRY(dalloc(c, (size_t)(n0 + 1) * 4, &h->roff, "delta rows per rank"));
    if (h->ds) {
      // target-major delta slots with whole words per target: y * nrank_d + rank
      const size_t nsd = (size_t)h->nrank_d * (size_t)h->range1, nwd = nsd / 32;
      XL_TRY(dalloc(c, nsd * 4, &h->dcur, "dense delta values"));
      XL_TRY(dalloc(c, nsd * 4, &h->dnext, "dense delta values"));
      XL_TRY(dalloc(c, nwd * 4, &h->dcur_pres, "dense delta bits"));
      XL_TRY(dalloc(c, nwd * 4, &h->dnext_pres, "dense delta bits"));
      XL_TRY(dalloc(c, nwd * 4, &h->dchg, "dense delta marks"));
      HIP_TRY(c, k::fill_bytes(h->dcur_pres.p, 0, nwd * 4, c->stream));
      HIP_TRY(c, k::fill_bytes(h->dnext_pres.p, 0, nwd * 4, c->stream));
      HIP_TRY(c, k::fill_bytes(h->dchg.p, 0, nwd * 4, c->stream));
    } else {
      XL_TRY(dalloc(c, ns * 4, &h->didx, "delta slot list"));
    }
    h->keys = 0;
    if (h->preloaded) {
      HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
      HIP_TRY(c, k::dense_insert_rows(h->dvals.as<uint32_t>(), h->dpres.as<uint32_t>(), h->dmap.as<uint32_t>(),
                                      range, (uint32_t)h->range1, r->col[0], h->nkey == 2 ? r->col[1] : nullptr,
                                      r->col[h->nkey], h->preloaded, h->kp, r->types[h->nkey],
                                      h->agg == Agg::MAX, c->dcounters, c->stream));
      u64 cnt[CNT_N];
      XL_TRY(ctl_read(c, c->dcounters, sizeof(cnt), cnt));
      if (cnt[CNT_FATAL]) return c->fail(XL_DEVICE_ERROR, "loaded row outside the dense domain (internal)");
      h->keys = (int64_t)cnt[CNT_INSERTED];
    }
    return XL_OK;
  }

  xl_status init_head(HeadRun* h) {
    Relation* r = h->rel;
    if (h->dv) {
      XL_TRY(init_dv(h));
      if (h->dv) return XL_OK;
    }
    if (h->dense) return init_dense(h);
    if (h->dcount) return init_dcount(h);
    h->cap = initial_cap(h->preloaded);
    XL_TRY(alloc_table(h, h->cap, &h->table));
    if (h->is_set) {
      h->rows_cap = h->cap;
      for (int j = 0; j < h->nkey; ++j) {
        XL_TRY(dalloc(c, (size_t)h->rows_cap * 4, &h->rows[j], "relation rows"));
        if (h->preloaded)
          HIP_TRY(c, hipMemcpyAsync(h->rows[j].p, r->col[j], (size_t)h->preloaded * 4,
                                    hipMemcpyDeviceToDevice, c->stream));
      }
      if (h->preloaded)
        HIP_TRY(c, k::set_insert_rows(h->table.as<u64>(), (u64)h->cap - 1, h->rows[0].as<uint32_t>(),
                                      h->nkey == 2 ? h->rows[1].as<uint32_t>() : nullptr, h->preloaded,
                                      h->kp, c->dcounters, c->stream));
      h->nrows = h->keys = h->preloaded;
      h->dbeg = h->dend = 0;
    } else {
      if (h->is_minmax) {
        XL_TRY(dalloc(c, (size_t)h->cap * 4, &h->didx, "delta slot list"));
        h->keys = 0;
        if (h->preloaded) {  // several loaded rows may share a key: count distinct keys
          HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
          HIP_TRY(c, k::table16_insert_rows(h->table.as<Slot16>(), (u64)h->cap - 1, r->col[0],
                                            h->nkey == 2 ? r->col[1] : nullptr, r->col[h->nkey],
                                            h->preloaded, h->kp, r->types[h->nkey],
                                            h->agg == Agg::MAX, c->dcounters, c->stream));
          u64 cnt[CNT_N];
          XL_TRY(ctl_read(c, c->dcounters, sizeof(cnt), cnt));
          if (cnt[CNT_FATAL]) return c->fail(XL_DEVICE_ERROR, "hash table probe exhausted (internal)");
          h->keys = (int64_t)cnt[CNT_INSERTED];
        }
      }
    }
    return XL_OK;
  }

  // Grow the head's table (and row list) so it holds at least `need` keys.
  xl_status grow(HeadRun* h, int64_t need) {
    int64_t ncap = h->cap * 4;
    while (ncap / 2 < need || ncap - need < WAVE_SLACK * 4 * EMIT_GRID + 1024) ncap *= 2;
    Buf nt;
    XL_TRY(alloc_table(h, ncap, &nt));
    HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
    if (h->is_set) {
      Buf nr[2];
      for (int j = 0; j < h->nkey; ++j) {
        XL_TRY(dalloc(c, (size_t)ncap * 4, &nr[j], "relation rows"));
        HIP_TRY(c, hipMemcpyAsync(nr[j].p, h->rows[j].p, (size_t)h->nrows * 4, hipMemcpyDeviceToDevice,
                                  c->stream));
      }
      HIP_TRY(c, k::set_insert_rows(nt.as<u64>(), (u64)ncap - 1, nr[0].as<uint32_t>(),
                                    h->nkey == 2 ? nr[1].as<uint32_t>() : nullptr, h->nrows, h->kp,
                                    c->dcounters, c->stream));
      for (int j = 0; j < h->nkey; ++j) std::swap(h->rows[j].p, nr[j].p);
      h->rows_cap = ncap;
    } else {
      HIP_TRY(c, k::table16_rehash(h->table.as<Slot16>(), h->cap, nt.as<Slot16>(), (u64)ncap - 1,
                                   c->dcounters, c->stream));
      if (h->is_minmax) {
        Buf nd;
        XL_TRY(dalloc(c, (size_t)ncap * 4, &nd, "delta slot list"));
        std::swap(h->didx.p, nd.p);
      }
    }
    std::swap(h->table.p, nt.p);
    h->cap = ncap;
    st->table_grows++;
    u64 cnt[CNT_N];
    XL_TRY(ctl_read(c, c->dcounters, sizeof(cnt), cnt));
    if (cnt[CNT_FATAL]) return c->fail(XL_DEVICE_ERROR, "hash table rebuild failed");
    if (h->is_minmax && h->didx_n > 0) {
      // the slots listed for the current round moved: list the slots stamped
      // with the round again (in slot order)
      Buf tmp, tot;
      XL_TRY(dalloc(c, k::compact_temp_bytes(h->cap), &tmp, "compaction scratch"));
      XL_TRY(dalloc(c, 8, &tot, "count"));
      HIP_TRY(c, k::table16_stamped(h->table.as<Slot16>(), h->cap, h->round, h->didx.as<uint32_t>(), h->cap,
                                    tot.as<uint32_t>(), tmp.p, c->stream));
      uint32_t n2 = 0;
      XL_TRY(ctl_read(c, tot.p, 4, &n2));
      h->didx_n = (int64_t)n2;
    }
    return XL_OK;
  }

  // ------------------------------------------------------------ rule evaluation
  struct Source {
    const uint32_t* col[MAXV];
    int64_t n;
  };

  Source resolve_driver(const RulePlan& p) {
    Source s{};
    HeadRun* h = head_of(p.driver);
    if (h && p.driver_delta) {
      if (h->is_set && !h->dense) {
        for (int j = 0; j < h->nkey; ++j) s.col[j] = h->rows[j].as<uint32_t>() + h->dbeg;
        s.n = h->dend - h->dbeg;
      } else {
        for (int j = 0; j < p.driver->arity; ++j) s.col[j] = h->drow[j].as<uint32_t>();
        s.n = h->dn;
      }
    } else if (h && h->is_set) {  // full scan of a head of this stratum (seed)
      for (int j = 0; j < h->nkey; ++j) s.col[j] = h->rows[j].as<uint32_t>();
      s.n = h->preloaded;
    } else {
      for (int j = 0; j < p.driver->arity; ++j) s.col[j] = p.driver->col[j];
      s.n = h ? h->preloaded : p.driver->nrows;
    }
    return s;
  }

  xl_status fill_ops(StageArgs& a, const RulePlan& p, int ks) {
    a.nops = (int)p.stage_ops[ks].size();
    for (int i = 0; i < a.nops; ++i) a.ops[i] = p.stage_ops[ks][i];
    for (size_t i = 0; i < p.stage_consts[ks].size(); ++i) a.consts[i] = p.stage_consts[ks][i];
    for (size_t q = 0; q < p.negs.size(); ++q) XL_TRY(get_neg(p.negs[q], &a.neg[q]));
    return XL_OK;
  }

  // The negation table of a negated literal over a complete relation (its
  // stratum ran before; stratification guarantees it): q's rows projected
  // onto the constrained columns, packed and radix sorted.
  xl_status get_neg(const NegPlan& np, NegTable* out) {
    for (auto& t : negtabs)
      if (t->rel == np.rel && t->ncols == np.ncols && (np.ncols < 1 || t->col[0] == np.col[0]) &&
          (np.ncols < 2 || t->col[1] == np.col[1])) {
        *out = NegTable{t->keys.as<unsigned long long>(), t->n};
        return XL_OK;
      }
    if (head_of(np.rel)) return c->fail(XL_DEVICE_ERROR, "negated relation is not complete (internal)");
    auto t = std::make_unique<DevNeg>();
    t->rel = np.rel;
    t->ncols = np.ncols;
    t->col[0] = np.col[0];
    t->col[1] = np.col[1];
    t->n = np.rel->nrows;
    if (np.ncols > 0 && t->n > 0) {
      Buf alt, tmp;
      XL_TRY(dalloc(c, (size_t)t->n * 8, &t->keys, "negation keys"));
      XL_TRY(dalloc(c, (size_t)t->n * 8, &alt, "negation keys"));
      XL_TRY(dalloc(c, k::radix_temp_bytes(t->n), &tmp, "sort scratch"));
      HIP_TRY(c, k::neg_keys(np.rel->col[np.col[0]], np.ncols > 1 ? np.rel->col[np.col[1]] : nullptr, t->n,
                             t->keys.as<u64>(), c->stream));
      int alt_used = 0;
      HIP_TRY(c, k::radix_sort_u64(t->keys.as<u64>(), nullptr, alt.as<u64>(), nullptr, t->n,
                                   np.ncols > 1 ? 64 : 32, tmp.p, c->stream, &alt_used));
      if (alt_used) std::swap(t->keys.p, alt.p);
    }
    *out = NegTable{t->keys.as<unsigned long long>(), t->n};
    negtabs.push_back(std::move(t));
    return XL_OK;
  }

  // Fatal flags of a stage launch: 32 is a join key with 2^26 or more rows
  // (the kernel's 32-bit match count per wavefront), anything else internal.
  xl_status stage_fatal(u64 flags, const char* internal) {
    if (flags & 32)
      return c->fail(XL_UNSUPPORTED, "a join key matches 2^26 or more rows of an indexed relation");
    return c->fail(XL_DEVICE_ERROR, internal);
  }

  xl_status counted_pass(StageArgs& a, int64_t* total, Buf* offs) {
    const int64_t nchunks = (a.src.n + 63) / 64;
    Buf cnt, tmp, tot;
    XL_TRY(dalloc(c, (size_t)nchunks * 8, &cnt, "chunk counts"));
    XL_TRY(dalloc(c, (size_t)nchunks * 8, offs, "chunk offsets"));
    XL_TRY(dalloc(c, k::scan_temp_bytes(nchunks), &tmp, "scan scratch"));
    XL_TRY(dalloc(c, 16, &tot, "count"));
    StageArgs ca = a;
    ca.emit.mode = EM_COUNT;
    ca.emit.chunk_cnt = cnt.as<u64>();
    ca.emit.counters = c->dcounters;
    HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
    HIP_TRY(c, k::stage_launch(ca, c->stream, 1 << 16));
    HIP_TRY(c, k::scan_exclusive_u64(cnt.as<u64>(), offs->as<u64>(), nchunks, tot.as<u64>(), tmp.p,
                                     c->stream));
    // the total and the fatal flags in one read
    HIP_TRY(c, hipMemcpyAsync(tot.as<u64>() + 1, c->dcounters + CNT_FATAL, 8, hipMemcpyDeviceToDevice, c->stream));
    u64 t[2] = {0, 0};
    XL_TRY(ctl_read(c, tot.p, 16, t));
    if (t[1]) return stage_fatal(t[1], "stage count pass failed (internal)");
    *total = (int64_t)t[0];
    return XL_OK;
  }

  // Kernel arguments of the closure-shaped variant in frontier form, reading
  // the current delta rows.
  xl_status frontier_args(const RulePlan& p, HeadRun* h, FrontierArgs& f) {
    f.x = h->fx.as<uint32_t>();
    f.in_cnt = h->fcnt[h->fcur].as<uint32_t>();
    f.in_diff = h->fdiff[h->fcur].as<uint32_t>();
    f.nseg = h->fn;
    XL_TRY(get_index(p.steps[0].rel, p.steps[0].key_col, &f.idx, -1, nullptr, 0, true));
    f.ybind_col = p.carried_ycol;
    f.bits = h->bits.as<uint32_t>();
    f.lo0 = h->kp.lo[0];
    f.lo1 = h->kp.lo[1];
    f.row_words = h->row_words;
    f.out_cnt = h->fcnt[h->fcur ^ 1].as<uint32_t>();
    f.out_diff = h->fdiff[h->fcur ^ 1].as<uint32_t>();
    f.pull_ratio = (uint32_t)c->pull_ratio;
    if (c->pull_ratio) {
      XL_TRY(get_index(p.steps[0].rel, p.carried_ycol, &f.rev, p.steps[0].key_col, &f.rev_first, 0, true));
      if (!f.rev_first) return c->fail(XL_DEVICE_ERROR, "pull index without first rows (internal)");
      f.rev_zcol = p.steps[0].key_col;
      if (!h->hasin.p) {
        XL_TRY(dalloc(c, (size_t)h->row_words * 4, &h->hasin, "in-edge bitmap"));
        HIP_TRY(c, k::hasin_bits(f.rev, h->kp.lo[1], h->row_words, h->hasin.as<uint32_t>(), c->stream));
      }
      f.hasin = h->hasin.as<uint32_t>();
    }
    f.counters = c->dcounters;
    return XL_OK;
  }

  // One gathered round: reads the delta rows flagged in gflag[gcur] from
  // (gcur ? gbits : dbits), writes the next delta into the other pair, then
  // clears the rows it read.
  xl_status gather_args(const RulePlan& p, HeadRun* h, GatherArgs& a) {
    GatherShape g;
    if (!gather_shape(p, &g)) return c->fail(XL_DEVICE_ERROR, "gathered round of another rule shape (internal)");
    a.in_bits = (h->gcur ? h->gbits : h->dbits).as<uint32_t>();
    a.out_bits = (h->gcur ? h->dbits : h->gbits).as<uint32_t>();
    a.in_flag = h->gflag[h->gcur].as<uint32_t>();
    a.out_flag = h->gflag[h->gcur ^ 1].as<uint32_t>();
    a.bits = h->bits.as<uint32_t>();
    XL_TRY(get_index(p.steps[g.s1].rel, g.x_col, &a.e1, -1, nullptr, 0, true));
    a.e1_acol = p.steps[g.s1].key_col;
    a.by_a = c->gather_rounds == 1;
    if (a.by_a) {
      XL_TRY(get_index(p.steps[g.s1].rel, a.e1_acol, &a.e1a, -1, nullptr, 0, true));
      a.e1_xcol = g.x_col;
      a.in_lo = h->gbound[h->gcur].as<uint32_t>();
      a.in_hi = a.in_lo + h->range0;
      a.out_lo = h->gbound[h->gcur ^ 1].as<uint32_t>();
      a.out_hi = a.out_lo + h->range0;
    }
    XL_TRY(get_index(p.steps[g.s2].rel, p.steps[g.s2].key_col, &a.push.idx, -1, nullptr, 0, true));
    a.push.ybind_col = g.y_col;
    a.lo0 = a.push.lo0 = h->kp.lo[0];
    a.lo1 = a.push.lo1 = h->kp.lo[1];
    a.row_words = a.push.row_words = h->row_words;
    a.range0 = h->range0;
    return XL_OK;
  }

  xl_status eval_gathered(const RulePlan& p, HeadRun* h) {
    h->fnew = 0;
    GatherArgs a{};
    XL_TRY(gather_args(p, h, a));
    a.counters = c->dcounters;
    HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
    if (c->profile) HIP_TRY(c, hipEventRecord(ev[0], c->stream));
    HIP_TRY(c, k::gather_round(a, c->stream));
    if (c->profile) HIP_TRY(c, hipEventRecord(ev[1], c->stream));
    // the consumed delta becomes the next round's output buffer (the by-row
    // kernel empties each delta row it reads itself)
    if (!a.by_a)
      HIP_TRY(c, k::clear_flagged_rows((h->gcur ? h->gbits : h->dbits).as<uint32_t>(),
                                       h->gflag[h->gcur].as<uint32_t>(), h->range0, h->row_words, nullptr, nullptr,
                                       c->stream));
    u64 cnt[CNT_N];
    XL_TRY(ctl_read(c, c->dcounters, sizeof(cnt), cnt));
    cands += (int64_t)cnt[CNT_CANDIDATES];
    if (c->profile) {
      float ms = 0;
      HIP_TRY(c, hipEventElapsedTime(&ms, ev[0], ev[1]));
      st->gather_ms += ms;
      st->gather_launches++;
      st->gather_candidates += (int64_t)cnt[CNT_CANDIDATES];
      st->gather_new += (int64_t)cnt[CNT_APPENDED];
    }
    h->fnew = (int64_t)cnt[CNT_APPENDED];
    h->keys += h->fnew;
    if (h->rel->max_rows > 0 && h->keys > h->rel->max_rows)
      return c->fail(XL_CAPACITY_EXCEEDED, "relation " + h->rel->name + " exceeds its max_rows " +
                                               std::to_string(h->rel->max_rows));
    return XL_OK;
  }

  // One round of the closure-shaped variant in frontier form.
  xl_status eval_frontier(const RulePlan& p, HeadRun* h) {
    h->fnew = 0;
    if (h->fn == 0) return XL_OK;
    FrontierArgs f{};
    XL_TRY(frontier_args(p, h, f));
    HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
    if (c->profile) HIP_TRY(c, hipEventRecord(ev[0], c->stream));
    HIP_TRY(c, k::frontier_round(f, c->stream));
    if (c->profile) HIP_TRY(c, hipEventRecord(ev[1], c->stream));
    u64 cnt[CNT_N];
    XL_TRY(ctl_read(c, c->dcounters, sizeof(cnt), cnt));
    cands += (int64_t)cnt[CNT_CANDIDATES];
    if (c->profile) {
      float ms = 0;
      HIP_TRY(c, hipEventElapsedTime(&ms, ev[0], ev[1]));
      st->front_ms += ms;
      st->front_launches++;
      st->front_candidates += (int64_t)cnt[CNT_CANDIDATES];
      st->front_new += (int64_t)cnt[CNT_APPENDED];
    }
    h->fnew = (int64_t)cnt[CNT_APPENDED];
    h->keys += h->fnew;
    if (h->rel->max_rows > 0 && h->keys > h->rel->max_rows)
      return c->fail(XL_CAPACITY_EXCEEDED, "relation " + h->rel->name + " exceeds its max_rows " +
                                               std::to_string(h->rel->max_rows));
    return XL_OK;
  }

  // Every pass of a frontier stratum in one launch (resident form): each
  // first key runs its own rounds until its delta is empty.  The pass count
  // and per-pass delta sizes match the round-by-round loop, since a key's
  // rounds never read another key's rows: the i-th pass's delta is the union
  // of every key's i-th round.
  bool resident_frontier(const Stratum& s) {
    return heads.size() == 1 && heads[0]->resident && heads[0]->frontier_ready &&
           s.variants.size() == 1 && s.variants[0].driver_delta && head_of(s.variants[0].head) == heads[0].get();
  }

  xl_status run_frontier_resident(const RulePlan& p, HeadRun* h, int64_t max_iterations) {
    if (h->fn == 0) return XL_OK;
    FrontierArgs f{};
    XL_TRY(frontier_args(p, h, f));
    f.x = nullptr;  // delta row sg of first key lo0 + sg is dbits row sg
    f.in_cnt = nullptr;
    f.in_diff = h->dbits.as<uint32_t>();
    f.nseg = h->range0;
    f.out_cnt = f.out_diff = nullptr;
    // one block, one read: the work queue, largest round and cap overflow in
    // a 256-byte block of their own (every workgroup's atomic on the queue
    // word is on the path to its next key, so no other counter shares its
    // cache line), the kernel's counters, then the new tuples of each round
    constexpr size_t HDR = 256, CNTB = 256, BLOCK = HDR + CNTB + 8 * XL_STATS_ROUNDS;
    static_assert(8 * CNT_N <= CNTB, "counters fit their block");
    Buf rs;
    XL_TRY(dalloc(c, BLOCK, &rs, "round counters"));
    HIP_TRY(c, hipMemsetAsync(rs.p, 0, BLOCK, c->stream));
    f.queue = rs.as<uint32_t>();
    f.max_round = rs.as<uint32_t>() + 1;
    f.overflow = rs.as<uint32_t>() + 2;
    f.counters = (unsigned long long*)((char*)rs.p + HDR);
    f.round_new = (unsigned long long*)((char*)rs.p + HDR + CNTB);
    f.round_slots = XL_STATS_ROUNDS;
    f.max_rounds = (uint32_t)std::min<int64_t>(max_iterations, 0xffffffffll);
    if (c->profile) HIP_TRY(c, hipEventRecord(ev[0], c->stream));
    HIP_TRY(c, k::frontier_resident(f, 0, c->stream));
    if (c->profile) HIP_TRY(c, hipEventRecord(ev[1], c->stream));
    std::vector<unsigned char> blk(BLOCK);
    XL_TRY(ctl_read(c, rs.p, BLOCK, blk.data()));
    uint32_t hdr[4];
    u64 cnt[CNT_N];
    memcpy(hdr, blk.data(), sizeof(hdr));
    memcpy(cnt, blk.data() + HDR, sizeof(cnt));
    const uint32_t rounds = hdr[1];
    std::vector<u64> per((size_t)XL_STATS_ROUNDS, 0);
    memcpy(per.data(), blk.data() + HDR + CNTB, 8 * (size_t)XL_STATS_ROUNDS);
    cands += (int64_t)cnt[CNT_CANDIDATES];
    if (c->profile) {
      float ms = 0;
      HIP_TRY(c, hipEventElapsedTime(&ms, ev[0], ev[1]));
      st->front_ms += ms;
      st->front_launches++;
      st->front_candidates += (int64_t)cnt[CNT_CANDIDATES];
      st->front_new += (int64_t)cnt[CNT_APPENDED];
    }
    // one recorded round per pass (the last counter slot sums the passes from
    // there on, which the receipt does not list anyway)
    for (uint32_t r = 0; r < rounds; ++r) {
      st->iterations++;
      record(r < (uint32_t)XL_STATS_ROUNDS ? (int64_t)per[r] : 0);
    }
    st->new_tuples_total += (int64_t)cnt[CNT_APPENDED];
    h->keys += (int64_t)cnt[CNT_APPENDED];
    h->fn = 0;
    if (hdr[2])
      return c->fail(XL_CONVERGENCE_FAILURE, "iteration cap " + std::to_string(max_iterations) +
                                                 " reached before the fixpoint");
    if (h->rel->max_rows > 0 && h->keys > h->rel->max_rows)
      return c->fail(XL_CAPACITY_EXCEEDED, "relation " + h->rel->name + " exceeds its max_rows " +
                                               std::to_string(h->rel->max_rows));
    return XL_OK;
  }

  // Turn the row-list delta [dbeg, dend) of a frontier head into delta bitmap
  // rows: sort by the first key, one delta row per distinct value.
  // First frontier: the seed round's new tuples are the delta bitmap; its
  // nonempty rows become the delta rows (no regrouping), then it is cleared.
  xl_status frontier_from_bits(HeadRun* h) {
    h->fn = 0;
    h->frontier_ready = true;
    if (h->round_new == 0) return XL_OK;
    Buf cnt, tmp, tot;
    XL_TRY(dalloc(c, (size_t)h->range0 * 4, &cnt, "row counts"));
    XL_TRY(dalloc(c, k::compact_temp_bytes(h->range0), &tmp, "compaction scratch"));
    XL_TRY(dalloc(c, 8, &tot, "count"));
    HIP_TRY(c, k::row_popcount(h->dbits.as<uint32_t>(), h->range0, h->row_words, cnt.as<uint32_t>(), c->stream));
    KeyPack kx{};
    kx.nkey = 1;
    kx.lo[0] = h->kp.lo[0];
    HIP_TRY(c, k::dcount_rows(cnt.as<uint32_t>(), h->range0, 1, kx, h->fx.as<uint32_t>(), nullptr,
                              h->fcnt[h->fcur].as<uint32_t>(), h->range0, tot.as<uint32_t>(), tmp.p, c->stream));
    uint32_t nseg = 0;
    XL_TRY(ctl_read(c, tot.p, 4, &nseg));
    HIP_TRY(c, k::gather_rows(h->dbits.as<uint32_t>(), h->row_words, h->fx.as<uint32_t>(), h->kp.lo[0], nseg,
                              h->fdiff[h->fcur].as<uint32_t>(), c->stream));
    HIP_TRY(c, k::fill_bytes(h->dbits.p, 0, (size_t)h->range0 * h->row_words * 4, c->stream));
    h->fn = nseg;
    return XL_OK;
  }



  // h(X, count(V)) :- r(..., X, ..., V, ...) with distinct variables, nothing
  // else in the body, over a finished relation that already has an index by
  // X's column: returns that index (the count per X is its degree), else null.
  const DevIndex* degree_index(const RulePlan& p) const {
    if (p.nkey != 1 || !p.steps.empty() || p.driver_delta) return nullptr;
    for (const auto& h : heads)
      if (h->rel == p.driver) return nullptr;
    for (const auto& ops : p.stage_ops)
      if (!ops.empty()) return nullptr;
    int kcol = -1;
    for (int j = 0; j < p.driver->arity; ++j) {
      const ColAct& a = p.driver_act[j];
      if (a.kind != CA_BIND && a.kind != CA_NONE) return nullptr;
      if (a.kind == CA_BIND && a.slot == p.key_slot[0]) {
        if (kcol >= 0) return nullptr;
        kcol = j;
      }
    }
    if (kcol < 0) return nullptr;
    for (const auto& ix : indexes)
      if (ix->rel == p.driver && ix->col == kcol && !ix->probe.keys) return ix.get();
    return nullptr;
  }

  // "value is P1 + W" / "P1 - W" with W bound by one column of e and nothing
  // else to check: returns 1 / 2 and the column, else 0.
  int affine_value(const RulePlan& p, int* col) const {
    const StepPlan& sp = p.steps[0];
    const auto& ops = p.stage_ops[0];
    if (p.cv_slot_p < 0 || ops.size() != 2) return 0;
    const MicroOp& m = ops[0];
    const MicroOp& o = ops[1];
    if (m.kind != OP_MOV || m.dst != p.val_slot || m.a != p.cv_slot_p || m.type != p.val_type) return 0;
    if ((o.kind != OP_ADD && o.kind != OP_SUB) || o.dst != p.val_slot || o.a != p.val_slot || o.b < 0 ||
        o.type != p.val_type)
      return 0;
    int wc = -1;
    for (int j = 0; j < sp.rel->arity; ++j) {
      const ColAct& ac = sp.act[j];
      if (ac.kind == CA_CHECK_SLOT || ac.kind == CA_CHECK_CONST) return 0;
      if (ac.kind == CA_BIND && ac.slot == o.b) wc = j;
    }
    if (wc < 0 || wc == sp.key_col || sp.rel->types[wc] != p.val_type) return 0;
    *col = wc;
    return o.kind == OP_ADD ? 1 : 2;
  }

  // One round of the carried-value variant over a dense sum/logsumexp head:
  // mark every key that receives a contribution (the stage kernel over the
  // delta rows), list the marked slots in order, then fold each key's
  // contributions by scanning e's rows for its Y value against the delta.
  // Arguments of the segmented pull of a carried-value rule over the current
  // delta (list, counts, row outputs and counters are set by the caller).
  xl_status pull_args(const RulePlan& p, HeadRun* h, int fast, int fcol, DensePullArgs& q) {
    const StepPlan& sp = p.steps[0];
    q.dict = h->dict.as<uint32_t>();
    q.range1 = (uint32_t)h->range1;
    q.nrank = (uint32_t)h->nrank_d;
    q.lo1 = h->kp.lo[1];
    XL_TRY(get_index(sp.rel, p.carried_ycol, &q.rev, -1, nullptr, 0, true));
    for (int j = 0; j < sp.rel->arity; ++j) q.rev.act[j] = sp.act[j];
    q.rev.act[p.carried_ycol].kind = CA_NONE;  // Y is bound from the key
    q.zcol = sp.key_col;
    q.slot_s = (int8_t)p.cv_slot_s;
    q.slot_z = (int8_t)p.cv_slot_z;
    q.slot_y = (int8_t)p.key_slot[1];
    q.slot_p = (int8_t)p.cv_slot_p;
    q.val_slot = (int8_t)p.val_slot;
    q.val_type = p.val_type;
    q.fold_kind = h->fold;
    q.fast = (int8_t)fast;
    q.fcol = (int8_t)fcol;
    q.nops = (int32_t)p.stage_ops[0].size();
    for (int i = 0; i < q.nops; ++i) q.ops[i] = p.stage_ops[0][i];
    for (size_t i = 0; i < p.stage_consts[0].size(); ++i) q.consts[i] = p.stage_consts[0][i];
    q.cval = h->dcur.as<uint32_t>();
    q.cpres = h->dcur_pres.as<uint32_t>();
    q.nval = h->dnext.as<uint32_t>();
    q.npres = h->dnext_pres.as<uint32_t>();
    q.fval = h->dvals.as<uint32_t>();
    q.fpres = h->dpres.as<uint32_t>();
    return XL_OK;
  }

  // Batched gathered rounds: each round gets its own counter block, so
  // `batched_rounds` rounds run per host read; rounds past the fixpoint find
  // no flagged delta row and change nothing.
  // ------------------------------------------------------------ batched set rounds
  // A recursive stratum with one set head held in a hash table (row list +
  // open-addressing set), whose delta variants each run in one stage-kernel
  // launch over the head's delta (one index step, or two fused into a
  // product) and join only relations outside the stratum, runs
  // batched_rounds rounds per host read: the head's row list is append-only,
  // so round j's delta is the rows between two boundaries that a one-thread
  // kernel records on the device after each round, and every launch reads
  // its driver range from there.  The batch shares one set of counters and
  // one load limit; a launch that crosses the limit (or refuses a product
  // row) sets the overflow flag, after which the rest of the batch does
  // nothing and the host re-runs that round the ordinary way (growing the
  // table; insert-if-absent keeps the partial round's rows valid).  Passes,
  // per-pass delta sizes and the iteration cap are those of the host loop.
  int batch_j = 0;              // round of the batch being enqueued (1-based; 0: not batching)
  // run by the next stage launch after the launch and before its count read
  std::function<xl_status()> before_count_read;
  int batch_grid = EMIT_GRID;  // workgroups of a batched launch (its waves bound the slack)
  // batched keyed value rounds: the batch's delta rows and slot list (one
  // position space: the first delta at [0, base), each round's slots and rows
  // after it), its capacity past the base, the round's stamp and the
  // accumulators of hashed folds
  uint32_t* batch_rows[3] = {nullptr, nullptr, nullptr};
  int64_t batch_rows_cap = 0;
  uint32_t* batch_idx = nullptr;
  u64 batch_delta_lim = 0;
  uint32_t batch_round = 0;
  u64* batch_acc = nullptr;

  // Batched rounds of set heads held in hash tables (row list + set): every
  // head of the stratum (one, or several in mutual recursion) is a hash set,
  // and each delta variant runs in one stage launch over its driver head's
  // delta and joins only relations outside the stratum.
  bool batched_sets(const Stratum& s) {
    if (c->batched_rounds <= 0 || heads.empty() || heads.size() > (size_t)k::MAX_BATCH_HEADS || s.variants.empty())
      return false;
    for (auto& hp : heads) {
      const HeadRun* h = hp.get();
      if (!h->is_set || h->dense || h->frontier || h->gathered || h->dv) return false;
    }
    for (const RulePlan& p : s.variants) {
      HeadRun* h = head_of(p.head);
      if (!p.driver_delta || !head_of(p.driver) || p.wcoj || !h) return false;
      for (const StepPlan& sp : p.steps)
        if (head_of(sp.rel)) return false;
      if (p.steps.size() > 2) return false;
      if (p.steps.size() == 2) {
        std::vector<MicroOp> pops;
        std::vector<uint32_t> pconsts;
        if (!c->product_joins || !product_plan(p, h, &pops, &pconsts)) return false;
      }
    }
    return true;
  }

  xl_status run_sets_batched(Stratum& s, int64_t max_iterations) {
    const int B = c->batched_rounds;
    const int nh = (int)heads.size();
    constexpr size_t CNTB = 256;
    static_assert(8 * CNT_N <= CNTB, "counters fit their block");
    const size_t per = CNTB + 8 * (size_t)(B + 2);  // one head's counters, then its round boundaries
    Buf blk;
    XL_TRY(dalloc(c, per * nh, &blk, "batch counters"));
    std::vector<unsigned char> host(per * nh);
    auto hcnt = [&](int q) { return (const u64*)(host.data() + per * q); };
    auto hbnd = [&](int q) { return (const u64*)(host.data() + per * q + CNTB); };
    for (int q = 0; q < nh; ++q) {
      heads[q]->b_cnt = (u64*)((char*)blk.p + per * q);
      heads[q]->b_bnd = (u64*)((char*)blk.p + per * q + CNTB);
    }
    auto any_delta = [&]() {
      for (auto& h : heads)
        if (h->dend > h->dbeg) return true;
      return false;
    };
    int64_t pass = 0;
    while (any_delta()) {
      if (pass >= max_iterations)
        return c->fail(XL_CONVERGENCE_FAILURE, "iteration cap " + std::to_string(max_iterations) +
                                                   " reached before the fixpoint");
      // every wavefront of a launch that crosses its head's limit may still
      // insert one batch: the grid takes at most a quarter of the smallest
      // table as slack (whatever the round's delta size, unknown here)
      int64_t waves = (int64_t)EMIT_GRID * 4;
      for (auto& h : heads) waves = std::min<int64_t>(waves, h->cap / 4 / WAVE_SLACK);
      waves = std::max<int64_t>(256, waves) / 4 * 4;
      batch_grid = (int)(waves / 4);
      bool grown = false;
      for (auto& hp : heads) {
        HeadRun* h = hp.get();
        const int64_t max_keys = std::min<int64_t>(h->cap / 2, h->cap - WAVE_SLACK * waves - 1024);
        if (h->keys >= max_keys) {
          XL_TRY(grow(h, std::max<int64_t>(h->keys * 2, h->keys + WAVE_SLACK * waves + 1024)));
          grown = true;
        }
        h->b_limit = (u64)std::max<int64_t>(0, max_keys - h->keys);
      }
      if (grown) continue;
      const int K = (int)std::min<int64_t>(B, max_iterations - pass);
      HIP_TRY(c, hipMemsetAsync(blk.p, 0, per * nh, c->stream));
      k::BatchMarks marks{};
      marks.n = nh;
      for (int q = 0; q < nh; ++q) {
        HeadRun* h = heads[q].get();
        HIP_TRY(c, k::batch_init(h->b_bnd, B + 2, (u64)h->dbeg, (u64)h->dend, c->stream));
        h->b_base = (u64)h->nrows;
        marks.bnd[q] = h->b_bnd;
        marks.cnt[q] = h->b_cnt;
        marks.base[q] = h->b_base;
      }
      if (c->profile) HIP_TRY(c, hipEventRecord(ev[0], c->stream));
      for (int j = 1; j <= K; ++j) {
        batch_j = j;
        for (RulePlan& p : s.variants) {
          const xl_status e = eval_plan(p);
          if (e != XL_OK) {
            batch_j = 0;
            return e;
          }
        }
        HIP_TRY(c, k::batch_mark_heads(marks, j, c->stream));
      }
      batch_j = 0;
      if (c->profile) HIP_TRY(c, hipEventRecord(ev[1], c->stream));
      XL_TRY(ctl_read(c, blk.p, per * nh, host.data()));
      u64 emitted = 0, candidates = 0;
      for (int q = 0; q < nh; ++q) {
        HeadRun* h = heads[q].get();
        const u64* cnt = hcnt(q);
        if (cnt[CNT_FATAL] & ~16ull)
          return stage_fatal(cnt[CNT_FATAL], "hash table probe exhausted or row list overflow (internal)");
        candidates += cnt[CNT_CANDIDATES];
        emitted += cnt[CNT_APPENDED];
        h->nrows = (int64_t)h->b_base + (int64_t)cnt[CNT_APPENDED];
        h->keys += (int64_t)cnt[CNT_APPENDED];
        if (h->rel->max_rows > 0 && h->keys > h->rel->max_rows)
          return c->fail(XL_CAPACITY_EXCEEDED, "relation " + h->rel->name + " exceeds its max_rows " +
                                                   std::to_string(h->rel->max_rows));
      }
      cands += (int64_t)candidates;
      if (c->profile) {
        float ms = 0;
        HIP_TRY(c, hipEventElapsedTime(&ms, ev[0], ev[1]));
        st->emit_ms += ms;
        st->emit_launches += (int64_t)K * (int64_t)s.variants.size();
        st->emit_candidates += (int64_t)candidates;
        st->emit_new += (int64_t)emitted;
      }
      // the marks are all or nothing: a round is complete for every head or for none
      int done = 0;
      bool empty = false;
      for (int j = 1; j <= K && hbnd(0)[j + 1] != ~0ull; ++j) {
        ++done;
        ++pass;
        st->iterations++;
        int64_t d = 0;
        for (int q = 0; q < nh; ++q) d += (int64_t)(hbnd(q)[j + 1] - hbnd(q)[j]);
        record(d);
        st->new_tuples_total += d;
        if (d == 0) {
          empty = true;
          break;
        }
      }
      if (empty) {
        for (auto& h : heads) h->dbeg = h->dend = h->nrows;
        break;
      }
      if (done == K) {
        for (int q = 0; q < nh; ++q) {
          heads[q]->dbeg = (int64_t)hbnd(q)[K];
          heads[q]->dend = (int64_t)hbnd(q)[K + 1];
        }
        continue;
      }
      // round done + 1 stopped early: re-run it the ordinary way (each head's
      // driver is [b[done], b[done + 1]); the rows its stopped launches
      // appended are the start of its delta, and insert-if-absent keeps them)
      if (pass >= max_iterations)
        return c->fail(XL_CONVERGENCE_FAILURE, "iteration cap " + std::to_string(max_iterations) +
                                                   " reached before the fixpoint");
      std::vector<int64_t> rb(nh);
      for (int q = 0; q < nh; ++q) {
        HeadRun* h = heads[q].get();
        rb[q] = (int64_t)hbnd(q)[done + 1];
        h->dbeg = (int64_t)hbnd(q)[done];
        h->dend = rb[q];
        begin_round(h);
      }
      for (RulePlan& p : s.variants) XL_TRY(eval_plan(p));
      ++pass;
      st->iterations++;
      int64_t d = 0;
      for (int q = 0; q < nh; ++q) {
        HeadRun* h = heads[q].get();
        d += h->nrows - rb[q];
        h->dbeg = rb[q];
        h->dend = h->nrows;
      }
      record(d);
      st->new_tuples_total += d;
    }
    return XL_OK;
  }

  // Batched rounds of a min/max or sum/logsumexp head held in a keyed hash
  // table (index mode 1, or key domains too wide for the dense forms): the
  // stratum's delta variants each run in one stage launch and join only
  // relations outside the stratum.  Min/max candidates improve table values
  // (EM_MINMAX); sum/logsumexp candidates fold into one accumulator per slot
  // (EM_HAGG).  Either way the slots a round touches are listed once (round
  // stamps) after the batch's earlier rounds, and a range kernel turns them
  // into the next delta rows at the same positions (for hashed folds it also
  // merges the round into the full relation and resets the accumulators),
  // so every size stays on the device until the batch's one read.
  bool batched_values(const Stratum& s) {
    if (c->batched_rounds <= 0 || heads.size() != 1 || s.variants.empty()) return false;
    HeadRun* h = heads[0].get();
    if (h->is_set || h->dense || h->dv || h->ds || h->tiled || h->frontier || h->gathered || h->dcount) return false;
    const int vt = h->rel->types[h->nkey];
    const bool hashed = h->is_sortagg && (h->fold == k::FOLD_SUM || h->fold == k::FOLD_LSE) &&
                        (vt == T_I32 || vt == T_F32);
    if (!h->is_minmax && !hashed) return false;
    for (const RulePlan& p : s.variants) {
      if (!p.driver_delta || p.driver != h->rel || p.wcoj || head_of(p.head) != h) return false;
      for (const StepPlan& sp : p.steps)
        if (head_of(sp.rel)) return false;
      if (p.steps.size() > 2) return false;
      if (p.steps.size() == 2) {
        std::vector<MicroOp> pops;
        std::vector<uint32_t> pconsts;
        if (!c->product_joins || !product_plan(p, h, &pops, &pconsts)) return false;
      }
    }
    return true;
  }

  // Copy n delta rows (key columns and value) from position `from` of the
  // columns src into the head's delta rows.
  xl_status take_delta_rows(HeadRun* h, uint32_t* const* src, int64_t from, int64_t n) {
    XL_TRY(ensure_drow(h, std::max<int64_t>(n, 1)));
    for (int j = 0; j <= h->nkey && n > 0; ++j)
      HIP_TRY(c, hipMemcpyAsync(h->drow[j].p, src[j] + from, (size_t)n * 4, hipMemcpyDeviceToDevice, c->stream));
    h->dn = n;
    return XL_OK;
  }

  xl_status run_values_batched(Stratum& s, HeadRun* h, int64_t max_iterations) {
    const int B = c->batched_rounds;
    const bool hashed = !h->is_minmax;
    const int vt = h->rel->types[h->nkey];
    constexpr size_t CNTB = 256;
    static_assert(8 * CNT_N <= CNTB, "counters fit their block");
    Buf blk;  // the batch's counters, then the round boundaries
    XL_TRY(dalloc(c, CNTB + 8 * (size_t)(B + 2), &blk, "batch counters"));
    u64* counters = blk.as<u64>();
    u64* bnd = (u64*)((char*)blk.p + CNTB);
    std::vector<unsigned char> host(CNTB + 8 * (size_t)(B + 2));
    Buf acc, bidx, brow[3];
    int64_t acc_cap = 0, bcap = 0;
    int64_t pass = 0;
    while (h->dn > 0) {
      if (pass >= max_iterations)
        return c->fail(XL_CONVERGENCE_FAILURE, "iteration cap " + std::to_string(max_iterations) +
                                                   " reached before the fixpoint");
      const int64_t waves =
          std::max<int64_t>(256, std::min<int64_t>((int64_t)EMIT_GRID * 4, h->cap / 4 / WAVE_SLACK)) / 4 * 4;
      batch_grid = (int)(waves / 4);
      const int64_t max_keys = std::min<int64_t>(h->cap / 2, h->cap - WAVE_SLACK * waves - 1024);
      if (h->keys >= max_keys) {
        XL_TRY(grow(h, std::max<int64_t>(h->keys * 2, h->keys + WAVE_SLACK * waves + 1024)));
        continue;
      }
      if (hashed && acc_cap != h->cap) {  // accumulators follow the table's slots (all at identity here)
        acc.reset();
        XL_TRY(dalloc(c, (size_t)h->cap * 8, &acc, "fold accumulators"));
        HIP_TRY(c, k::acc_fill(acc.as<u64>(), h->cap, vt, h->fold, c->stream));
        acc_cap = h->cap;
      }
      // a round touches each key at most once: the table's capacity past the
      // first delta holds a batch of typical rounds; more overflows the batch
      const int64_t need = h->dn + std::max<int64_t>(h->cap, 4096);
      if (bcap < need) {
        bidx.reset();
        XL_TRY(dalloc(c, (size_t)need * 4, &bidx, "batch delta slots"));
        for (int j = 0; j <= h->nkey; ++j) {
          brow[j].reset();
          XL_TRY(dalloc(c, (size_t)need * 4, &brow[j], "batch delta rows"));
        }
        bcap = need;
      }
      uint32_t* rows[3] = {brow[0].as<uint32_t>(), h->nkey == 2 ? brow[1].as<uint32_t>() : nullptr,
                           brow[h->nkey].as<uint32_t>()};
      uint32_t* cols[3] = {brow[0].as<uint32_t>(), brow[1].as<uint32_t>(), brow[2].as<uint32_t>()};
      for (int j = 0; j <= h->nkey; ++j)
        HIP_TRY(c, hipMemcpyAsync(brow[j].p, h->drow[j].p, (size_t)h->dn * 4, hipMemcpyDeviceToDevice, c->stream));
      const int K = (int)std::min<int64_t>(B, max_iterations - pass);
      const int64_t dn0 = h->dn;
      HIP_TRY(c, hipMemsetAsync(counters, 0, CNTB, c->stream));
      HIP_TRY(c, k::batch_init(bnd, B + 2, 0ull, (u64)dn0, c->stream));
      h->b_cnt = counters;
      h->b_bnd = bnd;
      h->b_base = (u64)dn0;
      h->b_limit = (u64)(max_keys - h->keys);
      for (int j = 0; j <= h->nkey; ++j) batch_rows[j] = brow[j].as<uint32_t>();
      batch_rows_cap = bcap;
      batch_idx = bidx.as<uint32_t>();
      batch_delta_lim = (u64)(bcap - dn0);
      batch_acc = hashed ? acc.as<u64>() : nullptr;
      if (c->profile) HIP_TRY(c, hipEventRecord(ev[0], c->stream));
      for (int j = 1; j <= K; ++j) {
        batch_j = j;
        batch_round = h->round + (uint32_t)j;
        for (RulePlan& p : s.variants) {
          const xl_status e = eval_plan(p);
          if (e != XL_OK) {
            batch_j = 0;
            return e;
          }
        }
        HIP_TRY(c, k::batch_mark(bnd, j, counters, (u64)dn0, c->stream));
        HIP_TRY(c, k::table16_rows_range(h->table.as<Slot16>(), batch_acc, bidx.as<uint32_t>(), bnd, j, bcap,
                                         h->kp, vt, h->fold, rows[0], rows[1], rows[2], c->stream));
      }
      batch_j = 0;
      batch_acc = nullptr;
      if (c->profile) HIP_TRY(c, hipEventRecord(ev[1], c->stream));
      XL_TRY(ctl_read(c, blk.p, CNTB + 8 * (size_t)(K + 2), host.data()));
      u64 cnt[CNT_N];
      memcpy(cnt, host.data(), sizeof(cnt));
      const u64* b = (const u64*)(host.data() + CNTB);
      if (cnt[CNT_FATAL] & ~16ull) return stage_fatal(cnt[CNT_FATAL], "hash table probe exhausted (internal)");
      cands += (int64_t)cnt[CNT_CANDIDATES];
      if (c->profile) {
        float ms = 0;
        HIP_TRY(c, hipEventElapsedTime(&ms, ev[0], ev[1]));
        st->emit_ms += ms;
        st->emit_launches += (int64_t)K * (int64_t)s.variants.size();
        st->emit_candidates += (int64_t)cnt[CNT_CANDIDATES];
        st->emit_new += (int64_t)cnt[CNT_INSERTED];
      }
      h->keys += (int64_t)cnt[CNT_INSERTED];
      if (h->rel->max_rows > 0 && h->keys > h->rel->max_rows)
        return c->fail(XL_CAPACITY_EXCEEDED, "relation " + h->rel->name + " exceeds its max_rows " +
                                                 std::to_string(h->rel->max_rows));
      int done = 0;
      bool empty = false;
      for (int j = 1; j <= K && b[j + 1] != ~0ull; ++j) {
        ++done;
        ++pass;
        st->iterations++;
        const int64_t d = (int64_t)(b[j + 1] - b[j]);
        record(d);
        st->new_tuples_total += d;
        if (d == 0) {
          empty = true;
          break;
        }
      }
      h->round += (uint32_t)done;
      if (empty) {
        h->dn = 0;
        break;
      }
      if (done == K) {  // the last round's rows are the next delta
        XL_TRY(take_delta_rows(h, cols, (int64_t)b[K], (int64_t)(b[K + 1] - b[K])));
        continue;
      }
      // Round done + 1 stopped early (table load limit, slot list capacity
      // or a refused product row): re-run it the ordinary way from its driver
      // rows [b[done], b[done + 1]).
      if (pass >= max_iterations)
        return c->fail(XL_CONVERGENCE_FAILURE, "iteration cap " + std::to_string(max_iterations) +
                                                   " reached before the fixpoint");
      XL_TRY(take_delta_rows(h, cols, (int64_t)b[done], (int64_t)(b[done + 1] - b[done])));
      const uint32_t rid = h->round + 1;  // the stopped round's stamp
      if (hashed) {
        // its contributions so far are dropped (the run below folds them all
        // again, under a new stamp, by the sorted path); keys it inserted
        // hold the identity until that run's merge
        HIP_TRY(c, k::acc_fill(acc.as<u64>(), acc_cap, vt, h->fold, c->stream));
        h->round = rid;
        begin_round(h);
      } else {
        // its improvements stay in the table: list the slots it stamped and
        // let the run below add the rest
        h->round = rid - 1;
        begin_round(h);
        Buf tmp, tot;
        XL_TRY(dalloc(c, k::compact_temp_bytes(h->cap), &tmp, "compaction scratch"));
        XL_TRY(dalloc(c, 8, &tot, "count"));
        HIP_TRY(c, k::table16_stamped(h->table.as<Slot16>(), h->cap, h->round, h->didx.as<uint32_t>(), h->cap,
                                      tot.as<uint32_t>(), tmp.p, c->stream));
        uint32_t n2 = 0;
        XL_TRY(ctl_read(c, tot.p, 4, &n2));
        h->didx_n = (int64_t)n2;
      }
      for (RulePlan& p : s.variants) XL_TRY(eval_plan(p));
      ++pass;
      st->iterations++;
      int64_t d = 0;
      XL_TRY(finish_round(h, &d));
      record(d);
      st->new_tuples_total += d;
    }
    return XL_OK;
  }

  bool batched_gather(const Stratum& s) {
    return c->batched_rounds > 0 && heads.size() == 1 && heads[0]->gathered && heads[0]->gather_ready &&
           s.variants.size() == 1 && s.variants[0].driver_delta && head_of(s.variants[0].head) == heads[0].get();
  }

  xl_status run_gather_batched(const RulePlan& p, HeadRun* h, int64_t max_iterations) {
    const int B = c->batched_rounds;
    Buf acc;
    XL_TRY(dalloc(c, (size_t)B * 8 * CNT_N, &acc, "round counters"));
    std::vector<hipEvent_t> evs;
    if (c->profile) {
      evs.resize(2 * (size_t)B, nullptr);
      for (auto& e : evs) HIP_TRY(c, hipEventCreate(&e));
    }
    auto destroy_events = [&]() {
      for (auto& e : evs)
        if (e) (void)hipEventDestroy(e);
      evs.clear();
    };
    int64_t pass = 0, delta = 1;
    xl_status status = XL_OK;
    while (delta > 0 && status == XL_OK) {
      if (pass >= max_iterations) {
        status = c->fail(XL_CONVERGENCE_FAILURE, "iteration cap " + std::to_string(max_iterations) +
                                                     " reached before the fixpoint");
        break;
      }
      const int nb = (int)std::min<int64_t>(B, max_iterations - pass);
      HIP_TRY(c, hipMemsetAsync(acc.p, 0, (size_t)nb * 8 * CNT_N, c->stream));
      for (int r = 0; r < nb; ++r) {
        GatherArgs a{};
        XL_TRY(gather_args(p, h, a));
        a.counters = acc.as<unsigned long long>() + (size_t)r * CNT_N;
        if (c->profile) HIP_TRY(c, hipEventRecord(evs[2 * r], c->stream));
        HIP_TRY(c, k::gather_round(a, c->stream));
        if (c->profile) HIP_TRY(c, hipEventRecord(evs[2 * r + 1], c->stream));
        if (!a.by_a)  // the by-row kernel empties each delta row it reads itself
          HIP_TRY(c, k::clear_flagged_rows((h->gcur ? h->gbits : h->dbits).as<uint32_t>(),
                                           h->gflag[h->gcur].as<uint32_t>(), h->range0, h->row_words, nullptr,
                                           nullptr, c->stream));
        h->gcur ^= 1;
      }
      std::vector<u64> cnt((size_t)nb * CNT_N);  // at most 64 blocks of 64 B: one control read
      XL_TRY(ctl_read(c, acc.p, (size_t)nb * 8 * CNT_N, cnt.data()));
      int done = nb;
      for (int r = 0; r < nb; ++r)
        if (cnt[(size_t)r * CNT_N + CNT_APPENDED] == 0) {
          done = r + 1;
          break;
        }
      for (int r = 0; r < done; ++r) {
        const u64* cr = cnt.data() + (size_t)r * CNT_N;
        st->iterations++;
        record((int64_t)cr[CNT_APPENDED]);
        st->new_tuples_total += (int64_t)cr[CNT_APPENDED];
        cands += (int64_t)cr[CNT_CANDIDATES];
        h->keys += (int64_t)cr[CNT_APPENDED];
        if (c->profile) {
          float ms = 0;
          HIP_TRY(c, hipEventElapsedTime(&ms, evs[2 * r], evs[2 * r + 1]));
          st->gather_ms += ms;
          st->gather_launches++;
          st->gather_candidates += (int64_t)cr[CNT_CANDIDATES];
          st->gather_new += (int64_t)cr[CNT_APPENDED];
        }
      }
      pass += done;
      delta = (int64_t)cnt[(size_t)(done - 1) * CNT_N + CNT_APPENDED];
    }
    destroy_events();
    if (status != XL_OK) return status;
    if (h->rel->max_rows > 0 && h->keys > h->rel->max_rows)
      return c->fail(XL_CAPACITY_EXCEEDED, "relation " + h->rel->name + " exceeds its max_rows " +
                                               std::to_string(h->rel->max_rows));
    return XL_OK;
  }

  // Batched pull rounds: a sum/logsumexp stratum whose one carried-value rule
  // adds or subtracts a column of e (every key with an in-edge from a delta
  // key gets a value, so the marks need no join) enqueues `batched_rounds`
  // rounds per host read.  Each round marks, lists and pulls with the key
  // count in device memory (the list holds every slot), writes no delta
  // rows, and leaves its delta size in a device array; rounds enqueued past
  // the fixpoint find no marks and change nothing.
  bool batched_pull(const Stratum& s) {
    if (c->batched_rounds <= 0 || heads.size() != 1 || !heads[0]->ds || s.variants.size() != 1 ||
        !s.variants[0].driver_delta || head_of(s.variants[0].head) != heads[0].get())
      return false;
    int fcol = 0;
    if (!affine_value(s.variants[0], &fcol)) return false;
    const HeadRun* h = heads[0].get();
    return (double)h->nrank_d * h->range1 * 4 <= (double)c->arena.largest_free() / 2;  // the list
  }

  xl_status run_pull_batched(const RulePlan& p, HeadRun* h, int64_t max_iterations) {
    const StepPlan& sp = p.steps[0];
    int fcol = 0;
    const int fast = affine_value(p, &fcol);
    const int64_t nsd = h->nrank_d * h->range1;
    IndexProbe fwd{};
    XL_TRY(get_index(sp.rel, sp.key_col, &fwd, -1, nullptr, 0, true));
    const int B = c->batched_rounds;
    Buf acc, rounds, list;
    XL_TRY(dalloc(c, 8 * CNT_N, &acc, "round counters"));
    XL_TRY(dalloc(c, (size_t)B * 4, &rounds, "round delta sizes"));
    XL_TRY(dalloc(c, (size_t)nsd * 4, &list, "marked keys"));
    HIP_TRY(c, hipMemsetAsync(acc.p, 0, 8 * CNT_N, c->stream));
    std::vector<hipEvent_t> evs;
    if (c->profile) {
      evs.resize(2 * (size_t)B, nullptr);
      for (auto& e : evs) HIP_TRY(c, hipEventCreate(&e));
    }
    auto destroy_events = [&]() {
      for (auto& e : evs)
        if (e) (void)hipEventDestroy(e);
      evs.clear();
    };
    int64_t pass = 0, delta = h->dn;
    xl_status status = XL_OK;
    while (delta > 0 && status == XL_OK) {
      if (pass >= max_iterations) {
        status = c->fail(XL_CONVERGENCE_FAILURE, "iteration cap " + std::to_string(max_iterations) +
                                                     " reached before the fixpoint");
        break;
      }
      const int nb = (int)std::min<int64_t>(B, max_iterations - pass);
      HIP_TRY(c, hipMemsetAsync(rounds.p, 0, (size_t)nb * 4, c->stream));
      for (int r = 0; r < nb; ++r) {
        uint32_t* nr = rounds.as<uint32_t>() + r;
        // the mark pass also clears the presence bits this round's pull
        // writes (the round before last's, no longer read)
        HIP_TRY(c, k::dense_mark_out(fwd, p.carried_ycol, h->kp.lo[1], (uint32_t)h->range1, (uint32_t)h->nrank_d,
                                     h->dcur_pres.as<uint32_t>(), h->dchg.as<uint32_t>(),
                                     h->dnext_pres.as<uint32_t>(), c->stream));
        HIP_TRY(c, k::bits_list_waves(h->dchg.as<uint32_t>(), nsd, list.as<uint32_t>(), nr, c->stream));
        DensePullArgs q{};
        XL_TRY(pull_args(p, h, fast, fcol, q));
        q.list = list.as<uint32_t>();
        q.n = nsd;
        q.n_dev = nr;
        q.counters = acc.as<unsigned long long>();
        if (c->profile) HIP_TRY(c, hipEventRecord(evs[2 * r], c->stream));
        HIP_TRY(c, k::dense_pull(q, c->stream));
        if (c->profile) HIP_TRY(c, hipEventRecord(evs[2 * r + 1], c->stream));
        std::swap(h->dcur.p, h->dnext.p);
        std::swap(h->dcur_pres.p, h->dnext_pres.p);
      }
      std::vector<uint32_t> n(nb);
      XL_TRY(ctl_read(c, rounds.p, (size_t)nb * 4, n.data()));
      int done = nb;
      for (int r = 0; r < nb; ++r)
        if (n[r] == 0) {
          done = r + 1;
          break;
        }
      for (int r = 0; r < done; ++r) {
        st->iterations++;
        record(n[r]);
        st->new_tuples_total += n[r];
        if (c->profile) {
          float ms = 0;
          HIP_TRY(c, hipEventElapsedTime(&ms, evs[2 * r], evs[2 * r + 1]));
          st->pull_ms += ms;
          st->pull_launches++;
          st->pull_new += n[r];
        }
      }
      pass += done;
      delta = n[done - 1];
    }
    destroy_events();
    // the next presence bits are clear between rounds everywhere else
    HIP_TRY(c, k::fill_bytes(h->dnext_pres.p, 0, (size_t)(nsd / 32) * 4, c->stream));
    u64 tot[CNT_N];
    XL_TRY(ctl_read(c, acc.p, sizeof(tot), tot));
    if (tot[CNT_FATAL]) return c->fail(XL_DEVICE_ERROR, "marked key without a contribution (internal)");
    cands += (int64_t)tot[CNT_CANDIDATES];
    if (c->profile) st->pull_candidates += (int64_t)tot[CNT_CANDIDATES];
    h->keys += (int64_t)tot[CNT_INSERTED];
    h->dn = 0;
    if (status != XL_OK) return status;
    if (h->rel->max_rows > 0 && h->keys > h->rel->max_rows)
      return c->fail(XL_CAPACITY_EXCEEDED, "relation " + h->rel->name + " exceeds its max_rows " +
                                               std::to_string(h->rel->max_rows));
    return XL_OK;
  }

  xl_status eval_dense_pull(const RulePlan& p, HeadRun* h) {
    h->pulled = true;
    h->pull_n = 0;
    Source src = resolve_driver(p);
    if (src.n == 0) return XL_OK;
    const StepPlan& sp = p.steps[0];
    StageArgs a{};
    a.src.n = src.n;
    a.src.ncols = p.driver->arity;
    for (int j = 0; j < a.src.ncols; ++j) {
      a.src.col[j] = src.col[j];
      a.src.act[j] = p.driver_act[j];
    }
    a.has_index = 1;
    XL_TRY(get_index(sp.rel, sp.key_col, &a.idx));
    a.idx.key_slot = (int8_t)sp.key_slot;
    for (int j = 0; j < sp.rel->arity; ++j) a.idx.act[j] = sp.act[j];
    XL_TRY(fill_ops(a, p, 0));
    int fcol = 0;
    const int fast = affine_value(p, &fcol);
    const int64_t nsd = h->nrank_d * h->range1;
    if (fast) {
      // every key with an in-edge from a delta key receives a value, so the
      // marks are the delta presence rows pushed to the out-neighbours (the
      // mark bits are clear: the previous list pass cleared what it listed)
      IndexProbe fwd{};
      XL_TRY(get_index(sp.rel, sp.key_col, &fwd, -1, nullptr, 0, true));
      if (c->profile) HIP_TRY(c, hipEventRecord(ev[0], c->stream));
      HIP_TRY(c, k::dense_mark_out(fwd, p.carried_ycol, h->kp.lo[1], (uint32_t)h->range1, (uint32_t)h->nrank_d,
                                   h->dcur_pres.as<uint32_t>(), h->dchg.as<uint32_t>(), nullptr, c->stream));
      if (c->profile) {
        HIP_TRY(c, hipEventRecord(ev[1], c->stream));
        HIP_TRY(c, hipEventSynchronize(ev[1]));
        float ms = 0;
        HIP_TRY(c, hipEventElapsedTime(&ms, ev[0], ev[1]));
        st->emit_ms += ms;
        st->emit_launches++;
        st->emit_source_rows += src.n;
      }
    }
    a.emit.mode = EM_MARK;
    a.emit.key.nkey = 2;
    a.emit.key.slot[0] = (int8_t)p.key_slot[0];
    a.emit.key.slot[1] = (int8_t)p.key_slot[1];
    a.emit.key.lo[0] = h->kp.lo[0];
    a.emit.key.lo[1] = h->kp.lo[1];
    a.emit.val_slot = (int8_t)p.val_slot;
    a.emit.dmap = h->dmap.as<uint32_t>();
    a.emit.dmap_n = (uint32_t)h->dmap_n;
    a.emit.row_bits = (u64)h->range1;
    a.emit.nrank = (uint32_t)h->nrank_d;
    a.emit.dchg = h->dchg.as<uint32_t>();
    a.emit.counters = c->dcounters;
    u64 cnt[CNT_N];
    if (!fast) {
      HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
      if (c->profile) HIP_TRY(c, hipEventRecord(ev[0], c->stream));
      HIP_TRY(c, k::stage_launch(a, c->stream, EMIT_GRID));
      if (c->profile) HIP_TRY(c, hipEventRecord(ev[1], c->stream));
      XL_TRY(ctl_read(c, c->dcounters, sizeof(cnt), cnt));
      if (cnt[CNT_FATAL]) return stage_fatal(cnt[CNT_FATAL], "key outside the dense domain (internal)");
      if (c->profile) {
        float ms = 0;
        HIP_TRY(c, hipEventElapsedTime(&ms, ev[0], ev[1]));
        st->emit_ms += ms;
        st->emit_launches++;
        st->emit_source_rows += src.n;
        st->emit_candidates += (int64_t)cnt[CNT_CANDIDATES];
      }
      cands += (int64_t)cnt[CNT_CANDIDATES];
    }
    const int64_t ns = nsd;
    Buf tmp, tot, list;
    XL_TRY(dalloc(c, k::bits_list_temp_bytes(ns), &tmp, "compaction scratch"));
    XL_TRY(dalloc(c, 8, &tot, "count"));
    HIP_TRY(c, k::bits_list(h->dchg.as<uint32_t>(), ns, nullptr, tot.as<uint32_t>(), tmp.p, false, c->stream));
    uint32_t n = 0;
    XL_TRY(ctl_read(c, tot.p, 4, &n));
    if (n == 0) return XL_OK;
    XL_TRY(dalloc(c, (size_t)n * 4, &list, "marked keys"));
    HIP_TRY(c, k::bits_list(h->dchg.as<uint32_t>(), ns, list.as<uint32_t>(), tot.as<uint32_t>(), tmp.p, true,
                            c->stream));
    for (int j = 0; j < 3; ++j) XL_TRY(dalloc(c, (size_t)n * 4, &h->ndrow[j], "delta rows"));
    DensePullArgs q{};
    XL_TRY(pull_args(p, h, fast, fcol, q));
    q.list = list.as<uint32_t>();
    q.n = n;
    q.k0 = h->ndrow[0].as<uint32_t>();
    q.k1 = h->ndrow[1].as<uint32_t>();
    q.v = h->ndrow[2].as<uint32_t>();
    q.counters = c->dcounters;
    HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
    if (c->profile) HIP_TRY(c, hipEventRecord(ev[0], c->stream));
    HIP_TRY(c, k::dense_pull(q, c->stream));
    if (c->profile) HIP_TRY(c, hipEventRecord(ev[1], c->stream));
    XL_TRY(ctl_read(c, c->dcounters, sizeof(cnt), cnt));
    if (cnt[CNT_FATAL]) return c->fail(XL_DEVICE_ERROR, "marked key without a contribution (internal)");
    if (c->profile) {
      float ms = 0;
      HIP_TRY(c, hipEventElapsedTime(&ms, ev[0], ev[1]));
      st->pull_ms += ms;
      st->pull_launches++;
      st->pull_candidates += (int64_t)cnt[CNT_CANDIDATES];
      st->pull_new += (int64_t)n;
    }
    if (fast) cands += (int64_t)cnt[CNT_CANDIDATES];  // no mark pass: count the in-edges the fold examined
    h->keys += (int64_t)cnt[CNT_INSERTED];
    h->pull_n = n;
    if (h->rel->max_rows > 0 && h->keys > h->rel->max_rows)
      return c->fail(XL_CAPACITY_EXCEEDED, "relation " + h->rel->name + " exceeds its max_rows " +
                                               std::to_string(h->rel->max_rows));
    return XL_OK;
  }

  // Tile layout (as many slots as fit 128 KB of LDS, or fewer so that every
  // CU gets a workgroup; a multiple of 32 slots) and e's rows sorted by
  // (tile of Y, Z) with offsets per (tile, Z): a tile's workgroup reads only
  // the rows that land in it, and one tile's rows of consecutive Z are
  // consecutive.
  xl_status build_tile_index(const RulePlan& p, HeadRun* h) {
    const StepPlan& sp = p.steps[0];
    Relation* e = sp.rel;
    const uint32_t max_tile = 32768;
    uint32_t nt = (uint32_t)((h->range1 + max_tile - 1) / max_tile);
    if (c->dense_tiles > 0) nt = (uint32_t)c->dense_tiles;
    else nt = std::max<uint32_t>(nt, (uint32_t)((256 + h->n0 - 1) / std::max<int64_t>(h->n0, 1)));
    uint32_t tile = (uint32_t)(((h->range1 + nt - 1) / nt + 31) / 32 * 32);
    tile = std::min<uint32_t>(std::max<uint32_t>(tile, 32), max_tile);
    h->tile = tile;
    h->ntiles = (uint32_t)((h->range1 + tile - 1) / tile);
    const int64_t n = e->nrows;
    IndexProbe& q = h->tidx;
    q = IndexProbe{};
    q.ncols = e->arity;
    const int zc = sp.key_col;
    const int64_t zr = n ? (int64_t)e->hi[zc] - e->lo[zc] + 1 : 0;
    const int64_t nkeys = zr * (h->ntiles + 1);
    if (nkeys >= ((int64_t)1 << 31)) return c->fail(XL_UNSUPPORTED, "tiled index key range too large");
    q.key_lo = n ? e->lo[zc] : 0;
    q.key_range = (uint32_t)zr;
    XL_TRY(dalloc(c, (size_t)(nkeys + 1) * 4, &h->toff, "tiled index offsets"));
    if (n == 0) {
      HIP_TRY(c, hipMemsetAsync(h->toff.p, 0, 4, c->stream));
      return XL_OK;
    }
    if (n > ((int64_t)1 << 30)) return c->fail(XL_UNSUPPORTED, "relation " + e->name + " too large to tile");
    // A loaded relation with Z in its first column and Y in its second is in
    // (Z, Y) order, so a stable sort by the tile of Y alone puts it in
    // (tile, Z) order when every Y lies in the head's domain; otherwise the
    // rows are sorted by the whole (tile, Z) key.
    const bool presorted = !head_of(e) && e->sorted && zc == 0 && p.carried_ycol == 1 && e->types[1] == T_I32 &&
                           (int64_t)e->lo[1] >= h->kp.lo[1] && (int64_t)e->hi[1] - h->kp.lo[1] < h->range1;
    Buf keys, keys2, perm, perm2, tmp;
    XL_TRY(dalloc(c, (size_t)n * 4, &keys, "index keys"));
    XL_TRY(dalloc(c, (size_t)n * 4, &keys2, "index keys"));
    XL_TRY(dalloc(c, (size_t)n * 4, &perm, "index permutation"));
    XL_TRY(dalloc(c, (size_t)n * 4, &perm2, "index permutation"));
    XL_TRY(dalloc(c, k::radix_temp_bytes(n), &tmp, "sort scratch"));
    HIP_TRY(c, k::tile_keys(e->col[zc], e->col[p.carried_ycol], n, e->lo[zc], h->kp.lo[1], h->tile, h->ntiles,
                            (uint32_t)zr, presorted, keys.as<uint32_t>(), c->stream));
    HIP_TRY(c, k::iota_u32(perm.as<uint32_t>(), n, c->stream));
    int alt = 0;
    const int key_bits = presorted ? bitlen((uint64_t)h->ntiles) : bitlen((uint64_t)nkeys - 1);
    HIP_TRY(c, k::radix_sort_u32(keys.as<uint32_t>(), perm.as<uint32_t>(), keys2.as<uint32_t>(), perm2.as<uint32_t>(),
                                 n, std::max(1, key_bits), tmp.p, c->stream, &alt));
    uint32_t* sk = alt ? keys2.as<uint32_t>() : keys.as<uint32_t>();
    uint32_t* spm = alt ? perm2.as<uint32_t>() : perm.as<uint32_t>();
    uint32_t* tc[MAXC] = {};
    for (int j = 0; j < e->arity; ++j) {
      h->tcols.push_back(std::make_unique<Buf>());
      XL_TRY(dalloc(c, (size_t)n * 4, h->tcols.back().get(), "tiled index column"));
      tc[j] = h->tcols.back()->as<uint32_t>();
      q.col[j] = tc[j];
    }
    HIP_TRY(c, k::gather_cols(e->col, tc, e->arity, spm, n, c->stream));
    if (presorted)  // the whole keys of the rows in their new order
      HIP_TRY(c, k::tile_keys(q.col[zc], q.col[p.carried_ycol], n, e->lo[zc], h->kp.lo[1], h->tile, h->ntiles,
                              (uint32_t)zr, false, sk, c->stream));
    HIP_TRY(c, k::csr_offsets(sk, n, (uint32_t)nkeys, h->toff.as<uint32_t>(), c->stream));
    return XL_OK;
  }

  // One round of the carried-value variant over a dense min/max head: one
  // workgroup per (rank, tile of second-key slots) with the tile in LDS.
  xl_status eval_dense_tiles(const RulePlan& p, HeadRun* h) {
    if (h->dn == 0) return XL_OK;
    DenseTileArgs a{};
    XL_TRY(tile_args(p, h, a));
    HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
    if (c->profile) HIP_TRY(c, hipEventRecord(ev[0], c->stream));
    HIP_TRY(c, k::dense_min_tiles(a, c->stream));
    if (c->profile) HIP_TRY(c, hipEventRecord(ev[1], c->stream));
    u64 cnt[CNT_N];
    XL_TRY(ctl_read(c, c->dcounters, sizeof(cnt), cnt));
    if (c->profile) {
      float ms = 0;
      HIP_TRY(c, hipEventElapsedTime(&ms, ev[0], ev[1]));
      st->emit_ms += ms;
      st->emit_launches++;
      st->emit_source_rows += h->dn;
      st->emit_candidates += (int64_t)cnt[CNT_CANDIDATES];
      st->emit_new += (int64_t)cnt[CNT_APPENDED];
    }
    cands += (int64_t)cnt[CNT_CANDIDATES];
    h->keys += (int64_t)cnt[CNT_INSERTED];
    if (h->rel->max_rows > 0 && h->keys > h->rel->max_rows)
      return c->fail(XL_CAPACITY_EXCEEDED, "relation " + h->rel->name + " exceeds its max_rows " +
                                               std::to_string(h->rel->max_rows));
    return XL_OK;
  }

  // Delta rows of a tiled head from its delta bits, grouped by rank (count
  // and write passes; the write pass also fills roff); the row total goes to
  // *total on the device.  With tcnt (the round's per-tile counts) one
  // launch that sums the counts itself replaces both passes.
  xl_status tile_delta_rows(HeadRun* h, uint32_t* total, Buf* ltmp, const uint32_t* tcnt) {
    if (tcnt) {
      HIP_TRY(c, k::tile_delta_rows(h->dchg.as<uint32_t>(), tcnt, (uint32_t)h->n0, h->ntiles, h->tile,
                                    (uint32_t)h->range1, h->dvals.as<uint32_t>(), h->dict.as<uint32_t>(), h->kp.lo[1],
                                    h->rel->types[h->nkey], h->fold, h->drow[0].as<uint32_t>(),
                                    h->drow[1].as<uint32_t>(), h->drow[2].as<uint32_t>(), h->roff.as<uint32_t>(),
                                    total, c->stream));
      return XL_OK;
    }
    const int64_t ns = std::max<int64_t>(h->n0, 1) * h->range1;
    for (bool write : {false, true})
      HIP_TRY(c, k::dense_delta_from_bits(h->dchg.as<uint32_t>(), ns, (uint32_t)h->range1, h->dvals.as<uint32_t>(),
                                          h->dict.as<uint32_t>(), h->kp.lo[1], h->rel->types[h->nkey], h->fold,
                                          h->drow[0].as<uint32_t>(), h->drow[1].as<uint32_t>(),
                                          h->drow[2].as<uint32_t>(), h->n0 > 0 ? h->roff.as<uint32_t>() : nullptr,
                                          total, ltmp->p, write, c->stream));
    return XL_OK;
  }

  // Tiled min/max stratum, rounds enqueued in batches (option
  // "batched_rounds"): every kernel of a round takes its sizes from device
  // memory (the rank offsets of the delta rows, the delta bits), the delta
  // row buffers hold any delta (one row per slot), and each round's delta
  // size goes to a device array that the host reads once per batch.  Rounds
  // enqueued past the fixpoint find an empty delta and change nothing, so
  // the pass count and per-pass sizes are the round-by-round ones.
  bool batched_tiles(const Stratum& s) {
    if (c->batched_rounds <= 0 || heads.size() != 1 || !heads[0]->tiled || s.variants.size() != 1 ||
        !s.variants[0].driver_delta || head_of(s.variants[0].head) != heads[0].get())
      return false;
    HeadRun* h = heads[0].get();
    const int64_t ns = std::max<int64_t>(h->n0, 1) * h->range1;
    return (double)ns * 12 <= (double)c->arena.largest_free() / 2;  // delta rows for every slot
  }

  xl_status run_tiles_batched(const RulePlan& p, HeadRun* h, int64_t max_iterations) {
    const int64_t ns = std::max<int64_t>(h->n0, 1) * h->range1;
    if (h->dcap < ns) {  // room for a delta row per slot, keeping the seed's rows
      Buf nd[3];
      for (int j = 0; j < 3; ++j) {
        XL_TRY(dalloc(c, (size_t)ns * 4, &nd[j], "delta rows"));
        if (h->dn)
          HIP_TRY(c, hipMemcpyAsync(nd[j].p, h->drow[j].p, (size_t)h->dn * 4, hipMemcpyDeviceToDevice, c->stream));
      }
      for (int j = 0; j < 3; ++j) {
        std::swap(h->drow[j].p, nd[j].p);
        h->drow[j].c = c;
      }
      h->dcap = ns;
    }
    DenseTileArgs a{};
    XL_TRY(tile_args(p, h, a));
    const int B = c->batched_rounds;
    Buf acc, rounds, ltmp, tcnt;
    XL_TRY(dalloc(c, 8 * CNT_N, &acc, "round counters"));
    XL_TRY(dalloc(c, (size_t)B * 4, &rounds, "round delta sizes"));
    XL_TRY(dalloc(c, k::bits_list_temp_bytes(ns), &ltmp, "compaction scratch"));
    // one-launch delta rows from per-tile counts when the tiles are few
    // enough for each listing workgroup to sum the counts before its tile
    const uint64_t nwork = (uint64_t)h->n0 * h->ntiles;
    if (h->n0 > 0 && nwork <= k::TL_MAX_WORK && h->tile <= k::TL_MAX_TILE && h->range1 % 32 == 0) {
      XL_TRY(dalloc(c, (size_t)nwork * 4, &tcnt, "tile delta counts"));
      a.tcnt = tcnt.as<uint32_t>();
    }
    HIP_TRY(c, hipMemsetAsync(acc.p, 0, 8 * CNT_N, c->stream));
    a.counters = acc.as<unsigned long long>();
    std::vector<hipEvent_t> evs;
    if (c->profile) {
      evs.resize(2 * (size_t)B, nullptr);
      for (auto& e : evs) HIP_TRY(c, hipEventCreate(&e));
    }
    auto destroy_events = [&]() {
      for (auto& e : evs)
        if (e) (void)hipEventDestroy(e);
      evs.clear();
    };
    int64_t pass = 0, delta = h->dn;
    xl_status status = XL_OK;
    while (delta > 0 && status == XL_OK) {
      if (pass >= max_iterations) {
        status = c->fail(XL_CONVERGENCE_FAILURE, "iteration cap " + std::to_string(max_iterations) +
                                                     " reached before the fixpoint");
        break;
      }
      const int nb = (int)std::min<int64_t>(B, max_iterations - pass);
      for (int r = 0; r < nb; ++r) {
        if (c->profile) HIP_TRY(c, hipEventRecord(evs[2 * r], c->stream));
        HIP_TRY(c, k::dense_min_tiles(a, c->stream));
        if (c->profile) HIP_TRY(c, hipEventRecord(evs[2 * r + 1], c->stream));
        XL_TRY(tile_delta_rows(h, rounds.as<uint32_t>() + r, &ltmp, a.tcnt));
      }
      std::vector<uint32_t> n(nb);
      XL_TRY(ctl_read(c, rounds.p, (size_t)nb * 4, n.data()));
      int done = nb;
      for (int r = 0; r < nb; ++r)
        if (n[r] == 0) {
          done = r + 1;
          break;
        }
      for (int r = 0; r < done; ++r) {
        st->iterations++;
        record(n[r]);
        st->new_tuples_total += n[r];
        if (c->profile) {
          float ms = 0;
          HIP_TRY(c, hipEventElapsedTime(&ms, evs[2 * r], evs[2 * r + 1]));
          st->emit_ms += ms;
          st->emit_launches++;
          st->emit_source_rows += r == 0 ? delta : n[r - 1];
        }
      }
      pass += done;
      delta = n[done - 1];
    }
    destroy_events();
    u64 tot[CNT_N];
    XL_TRY(ctl_read(c, acc.p, sizeof(tot), tot));
    cands += (int64_t)tot[CNT_CANDIDATES];
    if (c->profile) {
      st->emit_candidates += (int64_t)tot[CNT_CANDIDATES];
      st->emit_new += (int64_t)tot[CNT_APPENDED];
    }
    h->keys += (int64_t)tot[CNT_INSERTED];
    h->dn = 0;
    if (status != XL_OK) return status;
    if (h->rel->max_rows > 0 && h->keys > h->rel->max_rows)
      return c->fail(XL_CAPACITY_EXCEEDED, "relation " + h->rel->name + " exceeds its max_rows " +
                                               std::to_string(h->rel->max_rows));
    return XL_OK;
  }

  // Arguments of the tiled min/max round kernel for the current delta rows.
  xl_status tile_args(const RulePlan& p, HeadRun* h, DenseTileArgs& a) {
    const StepPlan& sp = p.steps[0];
    a.dk1 = h->drow[1].as<uint32_t>();
    a.dval = h->drow[2].as<uint32_t>();
    a.roff = h->roff.as<uint32_t>();
    a.dict = h->dict.as<uint32_t>();
    a.n0 = (uint32_t)h->n0;
    a.range1 = (uint32_t)h->range1;
    a.lo1 = h->kp.lo[1];
    if (!h->toff.p) XL_TRY(build_tile_index(p, h));
    a.tile = h->tile;
    a.ntiles = h->ntiles;
    a.idx = h->tidx;
    a.toff = h->toff.as<uint32_t>();
    for (int j = 0; j < sp.rel->arity; ++j) a.idx.act[j] = sp.act[j];
    a.ycol = p.carried_ycol;
    a.slot_s = (int8_t)p.cv_slot_s;
    a.slot_z = (int8_t)p.cv_slot_z;
    a.slot_p = (int8_t)p.cv_slot_p;
    a.slot_y = (int8_t)p.key_slot[1];
    a.val_slot = (int8_t)p.val_slot;
    a.val_type = p.val_type;
    a.is_max = h->agg == Agg::MAX;
    int fcol = 0;
    a.fast = (int8_t)affine_value(p, &fcol);
    a.fcol = (int8_t)fcol;
    a.nops = (int32_t)p.stage_ops[0].size();
    for (int i = 0; i < a.nops; ++i) a.ops[i] = p.stage_ops[0][i];
    for (size_t i = 0; i < p.stage_consts[0].size(); ++i) a.consts[i] = p.stage_consts[0][i];
    a.vals = h->dvals.as<uint32_t>();
    a.pres = h->dpres.as<uint32_t>();
    a.chg = h->dchg.as<uint32_t>();
    a.counters = c->dcounters;
    return XL_OK;
  }

  // Two index steps whose keys the driver row binds both (e.g. the children
  // of both members of a same-generation pair): one launch walks the product
  // of the two match lists, with both stages' micro-ops, instead of
  // materializing the first step's bindings.  Set heads only: a row whose
  // product is too long is refused by the kernel and the rule then runs
  // again with the two steps apart, which insert-if-absent makes harmless.
  bool product_plan(const RulePlan& p, const HeadRun* h, std::vector<MicroOp>* ops, std::vector<uint32_t>* consts) {
    if (p.steps.size() != 2 || !h->is_set || h->frontier) return false;
    const int k2 = p.steps[1].key_slot;
    bool by_driver = false;
    for (int j = 0; j < p.driver->arity; ++j)
      by_driver = by_driver || (p.driver_act[j].kind == CA_BIND && p.driver_act[j].slot == k2);
    if (!by_driver) return false;
    *ops = p.stage_ops[0];
    *consts = p.stage_consts[0];
    const int shift = (int)p.stage_consts[0].size();
    for (MicroOp op : p.stage_ops[1]) {
      if (op.a < 0) op.a = (int8_t)(op.a - shift);
      if (op.b < 0) op.b = (int8_t)(op.b - shift);
      ops->push_back(op);
    }
    for (uint32_t v : p.stage_consts[1]) consts->push_back(v);
    return ops->size() <= (size_t)MAXOPS && consts->size() <= (size_t)MAXK;
  }

  xl_status eval_plan(const RulePlan& p, bool allow_product = true) {
    HeadRun* h = head_of(p.head);
    if (h->frontier && p.driver_delta) return eval_frontier(p, h);
    if (h->gathered && p.driver_delta) return eval_gathered(p, h);
    if (h->ds && p.driver_delta) return eval_dense_pull(p, h);
    if (h->tiled && p.driver_delta) return eval_dense_tiles(p, h);
    const int nst = (int)p.steps.size();
    const int nkst = nst > 0 ? nst : 1;
    Source src = resolve_driver(p);
    HeadRun* hd = batch_j && p.driver_delta ? head_of(p.driver) : nullptr;
    if (hd) {  // batched rounds: the delta range is on the device
      if (hd->is_set) {
        for (int j = 0; j < hd->nkey; ++j) src.col[j] = hd->rows[j].as<uint32_t>();
        src.n = hd->rows_cap;  // bounds the grid only
      } else {
        for (int j = 0; j <= h->nkey; ++j) src.col[j] = batch_rows[j];
        src.n = batch_rows_cap;
      }
    }
    if (src.n == 0) return XL_OK;
    std::vector<MicroOp> pops;
    std::vector<uint32_t> pconsts;
    const bool product = allow_product && c->product_joins && product_plan(p, h, &pops, &pconsts);
    bool refused = false;
    // materialized bindings between stages
    std::vector<std::unique_ptr<Buf>> live_bufs;
    RowSource rs{};
    rs.n = src.n;
    rs.ncols = p.driver->arity;
    for (int j = 0; j < rs.ncols; ++j) {
      rs.col[j] = src.col[j];
      rs.act[j] = p.driver_act[j];
    }
    for (int ks = 0; ks < nkst; ++ks) {
      StageArgs a{};
      a.src = rs;
      a.has_index = nst > 0;
      if (nst > 0) {
        const StepPlan& sp = p.steps[ks];
        XL_TRY(get_index(sp.rel, sp.key_col, &a.idx));
        a.idx.key_slot = (int8_t)sp.key_slot;
        for (int j = 0; j < sp.rel->arity; ++j) a.idx.act[j] = sp.act[j];
      }
      XL_TRY(fill_ops(a, p, ks));
      if (product) {
        const StepPlan& s2 = p.steps[1];
        a.has_idx2 = 1;
        XL_TRY(get_index(s2.rel, s2.key_col, &a.idx2));
        a.idx2.key_slot = (int8_t)s2.key_slot;
        for (int j = 0; j < s2.rel->arity; ++j) a.idx2.act[j] = s2.act[j];
        a.nops = (int)pops.size();
        for (int i = 0; i < a.nops; ++i) a.ops[i] = pops[i];
        for (size_t i = 0; i < pconsts.size(); ++i) a.consts[i] = pconsts[i];
      }
      a.emit.counters = c->dcounters;
      if (!product && ks + 1 < nkst) {
        // intermediate: count -> scan -> materialize the live slots
        const std::vector<int>& live = p.live_after[ks];
        a.emit.mode = EM_MAT;
        a.emit.nout = (int)live.size();
        int64_t total = 0;
        Buf offs;
        XL_TRY(counted_pass(a, &total, &offs));
        RowSource next{};
        next.n = total;
        next.ncols = (int)live.size();
        for (size_t q = 0; q < live.size(); ++q) {
          live_bufs.push_back(std::make_unique<Buf>());
          XL_TRY(dalloc(c, (size_t)std::max<int64_t>(total, 1) * 4, live_bufs.back().get(), "join bindings"));
          a.emit.out_slot[q] = (int8_t)live[q];
          a.emit.out_col[q] = live_bufs.back()->as<uint32_t>();
          next.col[q] = a.emit.out_col[q];
          next.act[q].kind = CA_BIND;
          next.act[q].slot = (int8_t)live[q];
        }
        a.emit.chunk_off = offs.as<u64>();
        a.emit.mat_base = 0;
        if (total > 0) HIP_TRY(c, k::stage_launch(a, c->stream, 1 << 16));
        rs = next;
        if (total == 0) return XL_OK;
        continue;
      }
      // final stage: emit into the head
      a.emit.key.nkey = p.nkey;
      a.emit.key.slot[0] = (int8_t)p.key_slot[0];
      a.emit.key.slot[1] = (int8_t)(p.nkey == 2 ? p.key_slot[1] : p.key_slot[0]);
      a.emit.key.lo[0] = h->kp.lo[0];
      a.emit.key.lo[1] = h->kp.lo[1];
      a.emit.key.shift = h->kp.shift;
      a.emit.val_slot = (int8_t)p.val_slot;
      a.emit.val_type = p.val_type;
      if (hd) {
        // batched rounds: the driver's delta range, the target's append base,
        // load limit and counters belong to the batch; nothing is read back
        a.src_range = hd->b_bnd + (batch_j - 1);
        a.emit.counters = h->b_cnt;
        a.emit.limit = h->b_limit;
        a.emit.mask = (u64)h->cap - 1;
        if (h->is_set) {
          a.emit.mode = EM_SET;
          a.emit.table = h->table.as<u64>();
          a.emit.row_col[0] = h->rows[0].as<uint32_t>();
          a.emit.row_col[1] = h->nkey == 2 ? h->rows[1].as<uint32_t>() : h->rows[0].as<uint32_t>();
          a.emit.row_base = h->b_base;
          a.emit.row_cap = h->rows_cap;
        } else {
          a.emit.mode = h->is_minmax ? EM_MINMAX : EM_HAGG;
          a.emit.table16 = h->table.as<Slot16>();
          a.emit.is_max = h->agg == Agg::MAX;
          a.emit.round = batch_round;
          a.emit.delta_idx = batch_idx + h->b_base;
          a.emit.delta_lim = batch_delta_lim;
          a.emit.acc = batch_acc;
          a.emit.fold_kind = h->fold;
          a.emit.agg_identity = h->fold == k::FOLD_LSE ? 0xff800000u : 0u;  // -inf, or zero
        }
        HIP_TRY(c, k::stage_launch(a, c->stream, batch_grid));
        if (product) break;  // the one launch covered both steps
        continue;
      }
      if (h->dcount) {
        const DevIndex* dx = degree_index(p);
        if (dx) {  // the group's count is the index degree of its key
          HIP_TRY(c, k::index_degree_add(dx->probe.off, dx->probe.key_range, dx->probe.key_lo, h->kp.lo[0],
                                         (uint32_t)h->range0, h->counts.as<uint32_t>(), c->dcheck, c->stream));
          cands += src.n;
          return XL_OK;
        }
        a.emit.mode = EM_DCOUNT;
        a.emit.bits = h->counts.as<uint32_t>();
        a.emit.row_bits = (u64)h->range1;
        HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
        HIP_TRY(c, k::stage_launch(a, c->stream, 1 << 16));
        u64 cnt[CNT_N];
        XL_TRY(ctl_read(c, c->dcounters, sizeof(cnt), cnt));
        if (cnt[CNT_FATAL]) return stage_fatal(cnt[CNT_FATAL], "count key outside the head domain (internal)");
        cands += (int64_t)cnt[CNT_CANDIDATES];
        return XL_OK;
      }
      if (h->is_sortagg) {
        a.emit.mode = EM_MAT;
        a.emit.mat_packed = 1;
        int64_t total = 0;
        Buf offs;
        XL_TRY(counted_pass(a, &total, &offs));
        cands += total;
        if (total == 0) return XL_OK;
        const size_t kb = key_bytes(h);
        if (h->cn + total > h->ccap) {
          const int64_t ncap = std::max<int64_t>(h->cn + total, h->ccap * 2);
          Buf nk, nv;
          XL_TRY(dalloc(c, (size_t)ncap * kb, &nk, "aggregate candidates"));
          XL_TRY(dalloc(c, (size_t)ncap * 4, &nv, "aggregate candidates"));
          if (h->cn) {
            HIP_TRY(c, hipMemcpyAsync(nk.p, h->ckey.p, (size_t)h->cn * kb, hipMemcpyDeviceToDevice, c->stream));
            HIP_TRY(c, hipMemcpyAsync(nv.p, h->cval.p, (size_t)h->cn * 4, hipMemcpyDeviceToDevice, c->stream));
          }
          std::swap(h->ckey.p, nk.p);
          std::swap(h->cval.p, nv.p);
          h->ckey.c = h->cval.c = c;
          h->ccap = ncap;
        }
        a.emit.out_key = h->ckey.as<u64>();
        a.emit.key32 = kb == 4;
        a.emit.out_val = h->cval.as<uint32_t>();
        a.emit.chunk_off = offs.as<u64>();
        a.emit.mat_base = h->cn;
        HIP_TRY(c, k::stage_launch(a, c->stream, 1 << 16));
        h->cn += total;
        return XL_OK;
      }
      // set / min / max: single pass with insert-or-improve, retried after growth
      for (int attempt = 0;; ++attempt) {
        if (attempt > 8) return c->fail(XL_DEVICE_ERROR, "hash table growth did not converge");
        if (nst == 0 || ks == 0) {  // the driver may live in this head's row list
          Source s2 = resolve_driver(p);
          for (int j = 0; j < a.src.ncols && ks == 0; ++j) a.src.col[j] = s2.col[j];
        }
        // Every wavefront may insert one more batch of 64 keys after the load
        // limit is crossed, so the limit leaves room for all of them: the
        // table can never fill and the row list never overflows.
        const int64_t waves = std::min<int64_t>((a.src.n + 63) / 64, (int64_t)EMIT_GRID * 4);
        if (h->dv) {  // every slot exists up front: nothing can overflow
          HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
          a.emit.limit = ~0ull;
          a.emit.mode = EM_DMIN;
          a.emit.bits = h->dvals.as<uint32_t>();
          a.emit.row_bits = (u64)h->range1;
          a.emit.dmap = h->dmap.as<uint32_t>();
          a.emit.dmap_n = (uint32_t)h->dmap_n;
          a.emit.dpres = h->dpres.as<uint32_t>();
          a.emit.dchg = h->dchg.as<uint32_t>();
          a.emit.is_max = h->agg == Agg::MAX;
          a.emit.delta_idx = h->didx.as<uint32_t>() + h->didx_n;
        } else if (h->dense) {  // bitmap and delta bitmap cover the whole domain
          HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
          a.emit.limit = ~0ull;
          a.emit.mode = EM_BITSET;
          a.emit.bits = h->bits.as<uint32_t>();
          a.emit.row_bits = h->row_bits;
          a.emit.dchg = h->dbits.as<uint32_t>();
        } else {
        const int64_t max_keys = std::min<int64_t>(h->cap / 2, h->cap - WAVE_SLACK * waves - 1024);
        if (h->keys >= max_keys) {
          XL_TRY(grow(h, std::max<int64_t>(h->keys * 2, h->keys + WAVE_SLACK * waves + 1024)));
          continue;
        }
        HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
        a.emit.limit = (u64)(max_keys - h->keys);
        a.emit.mask = (u64)h->cap - 1;
        }
        if (h->dense || h->dv) {
          // EM_BITSET / EM_DMIN configured above
        } else if (h->is_set) {
          a.emit.mode = EM_SET;
          a.emit.table = h->table.as<u64>();
          a.emit.row_col[0] = h->rows[0].as<uint32_t>();
          a.emit.row_col[1] = h->nkey == 2 ? h->rows[1].as<uint32_t>() : h->rows[0].as<uint32_t>();
          a.emit.row_base = h->nrows;
          a.emit.row_cap = h->rows_cap;
        } else {
          a.emit.mode = EM_MINMAX;
          a.emit.table16 = h->table.as<Slot16>();
          a.emit.is_max = h->agg == Agg::MAX;
          a.emit.round = h->round;
          a.emit.delta_idx = h->didx.as<uint32_t>() + h->didx_n;
        }
        if (c->profile) HIP_TRY(c, hipEventRecord(ev[0], c->stream));
        HIP_TRY(c, k::stage_launch(a, c->stream, EMIT_GRID));
        if (c->profile) HIP_TRY(c, hipEventRecord(ev[1], c->stream));
        if (before_count_read) {  // work that does not need this launch's counts, enqueued before waiting for them
          const auto f = std::move(before_count_read);
          before_count_read = nullptr;
          XL_TRY(f());
        }
        u64 cnt[CNT_N];
        XL_TRY(ctl_read(c, c->dcounters, sizeof(cnt), cnt));
        if (c->profile) {
          float ms = 0;
          HIP_TRY(c, hipEventElapsedTime(&ms, ev[0], ev[1]));
          st->emit_ms += ms;
          st->emit_launches++;
          st->emit_source_rows += a.src.n;
          st->emit_candidates += (int64_t)cnt[CNT_CANDIDATES];
          st->emit_new += (int64_t)(h->is_set ? cnt[CNT_APPENDED] : cnt[CNT_INSERTED] + cnt[CNT_APPENDED]);
        }
        if (product && cnt[CNT_FATAL] == 16) {
          refused = true;  // some product rows were skipped: the rule runs again unfused below
        } else if (cnt[CNT_FATAL]) {
          return stage_fatal(cnt[CNT_FATAL], h->dv ? "key outside the dense domain (internal)"
                                                   : "hash table probe exhausted or row list overflow (internal)");
        }
        cands += (int64_t)cnt[CNT_CANDIDATES];
        if (h->dense) {
          h->keys += (int64_t)cnt[CNT_APPENDED];
          h->round_new += (int64_t)cnt[CNT_APPENDED];
        } else if (h->is_set) {
          h->nrows += (int64_t)cnt[CNT_APPENDED];
          h->keys += (int64_t)cnt[CNT_APPENDED];
        } else {
          h->keys += (int64_t)cnt[CNT_INSERTED];
          h->didx_n += (int64_t)cnt[CNT_APPENDED];
        }
        if (h->rel->max_rows > 0 && h->keys > h->rel->max_rows)
          return c->fail(XL_CAPACITY_EXCEEDED, "relation " + h->rel->name + " exceeds its max_rows " +
                                                   std::to_string(h->rel->max_rows));
        if (!cnt[CNT_OVERFLOW]) break;
        XL_TRY(grow(h, h->keys * 2 + 1));  // (lists this round's min/max slots again)
      }
      if (product) break;  // the one launch covered both steps
    }
    if (refused) return eval_plan(p, false);
    return XL_OK;
  }

  // Candidate keys of sorted aggregation are 32-bit when the packed key fits.
  size_t key_bytes(const HeadRun* h) const {
    const int kbits = h->nkey == 2 ? h->bits0 + h->kp.shift : h->bits0;
    return kbits <= 32 ? 4 : 8;
  }

  xl_status ensure_drow(HeadRun* h, int64_t n) {
    if (n <= h->dcap) return XL_OK;
    const int64_t ncap = std::max<int64_t>(n, h->dcap * 2);
    for (int j = 0; j <= h->nkey; ++j) XL_TRY(dalloc(c, (size_t)ncap * 4, &h->drow[j], "delta rows"));
    h->dcap = ncap;
    return XL_OK;
  }

  void begin_round(HeadRun* h) {
    h->round++;
    h->round_new = 0;
    h->round_begin = h->nrows;
    h->didx_n = 0;
    h->cn = 0;
  }

  xl_status finish_round(HeadRun* h, int64_t* delta) {
    if (h->frontier && h->frontier_ready) {  // a frontier round produced the new delta rows
      h->fcur ^= 1;
      *delta = h->fnew;
      return XL_OK;
    }
    if (h->gathered && h->gather_ready) {  // a gathered round wrote the next delta rows
      h->gcur ^= 1;
      *delta = h->fnew;
      return XL_OK;
    }
    if (h->dense) {
      *delta = h->round_new;
      if (h->gathered) {  // seed round: its new tuples in dbits are the first delta rows
        h->gather_ready = true;
        h->gcur = 0;
        if (h->round_new) {
          HIP_TRY(c, k::row_popcount(h->dbits.as<uint32_t>(), h->range0, h->row_words, h->gflag[0].as<uint32_t>(),
                                     c->stream));
          // the seed's delta rows may hold bits anywhere
          HIP_TRY(c, k::fill_bounds(h->gbound[0].as<uint32_t>(), h->gbound[0].as<uint32_t>() + h->range0, h->range0,
                                    0u, (uint32_t)h->row_words, c->stream));
        }
        return XL_OK;
      }
      if (h->resident) {  // the resident launch reads the seed's delta rows from dbits
        h->frontier_ready = true;
        h->fn = h->round_new ? h->range0 : 0;
        return XL_OK;
      }
      if (h->frontier) return frontier_from_bits(h);  // seed round -> first frontier
      // this round's new tuples, in key order, become the delta rows
      const int64_t nbits = (int64_t)(h->nkey == 2 ? (u64)h->range0 * h->row_bits : (u64)((h->range0 + 31) / 32) * 32);
      Buf tmp, tot;
      XL_TRY(dalloc(c, k::bits_list_temp_bytes(nbits), &tmp, "compaction scratch"));
      XL_TRY(dalloc(c, 8, &tot, "count"));
      auto keys = [&](bool write) {
        return k::bits_keys(h->dbits.as<uint32_t>(), nbits, h->row_bits, h->kp.lo[0], h->kp.lo[1], h->nkey, true,
                            h->drow[0].as<uint32_t>(), h->nkey == 2 ? h->drow[1].as<uint32_t>() : nullptr,
                            tot.as<uint32_t>(), tmp.p, write, c->stream);
      };
      HIP_TRY(c, keys(false));
      uint32_t n = 0;
      XL_TRY(ctl_read(c, tot.p, 4, &n));
      if ((int64_t)n != h->round_new) return c->fail(XL_DEVICE_ERROR, "delta bitmap count mismatch (internal)");
      XL_TRY(ensure_drow(h, n));
      if (n) HIP_TRY(c, keys(true));
      h->dn = n;
      return XL_OK;
    }
    if (h->is_set) {
      h->dbeg = h->round_begin;
      h->dend = h->nrows;
      *delta = h->dend - h->dbeg;
      return XL_OK;
    }
    if (h->dcount) {
      *delta = 0;
      return XL_OK;  // counted in place; rows are produced at materialization
    }
    if (h->ds && h->pulled) {  // the pull wrote the next delta rows and values
      h->pulled = false;
      for (int j = 0; j < 3; ++j) {
        std::swap(h->drow[j].p, h->ndrow[j].p);
        h->drow[j].c = c;
        h->ndrow[j].reset();
      }
      h->dcap = h->pull_n;
      h->dn = h->pull_n;
      std::swap(h->dcur.p, h->dnext.p);
      std::swap(h->dcur_pres.p, h->dnext_pres.p);
      HIP_TRY(c, k::fill_bytes(h->dnext_pres.p, 0, (size_t)(h->nrank_d * h->range1 / 32) * 4, c->stream));
      *delta = h->dn;
      return XL_OK;
    }
    if (h->tiled) {  // delta rows from the delta bits, grouped by rank (the write pass fills roff)
      const int64_t ns = std::max<int64_t>(h->n0, 1) * h->range1;
      Buf ltmp, tot;
      XL_TRY(dalloc(c, k::bits_list_temp_bytes(ns), &ltmp, "compaction scratch"));
      XL_TRY(dalloc(c, 8, &tot, "count"));
      auto rows = [&](bool write) {
        return k::dense_delta_from_bits(h->dchg.as<uint32_t>(), ns, (uint32_t)h->range1, h->dvals.as<uint32_t>(),
                                   h->dict.as<uint32_t>(), h->kp.lo[1], h->rel->types[h->nkey], h->fold,
                                   h->drow[0].as<uint32_t>(), h->drow[1].as<uint32_t>(), h->drow[2].as<uint32_t>(),
                                   h->n0 > 0 ? h->roff.as<uint32_t>() : nullptr, tot.as<uint32_t>(), ltmp.p, write,
                                   c->stream);
      };
      HIP_TRY(c, rows(false));
      uint32_t n = 0;
      XL_TRY(ctl_read(c, tot.p, 4, &n));
      XL_TRY(ensure_drow(h, n));
      if (n) HIP_TRY(c, rows(true));
      h->dn = n;
      *delta = n;
      return XL_OK;
    }
    if (h->dv && !h->ds) {
      XL_TRY(ensure_drow(h, h->didx_n));
      HIP_TRY(c, k::dense_delta_rows(h->didx.as<uint32_t>(), h->didx_n, h->dvals.as<uint32_t>(),
                                     h->dchg.as<uint32_t>(), h->dict.as<uint32_t>(), (uint32_t)h->range1,
                                     h->kp.lo[1], h->rel->types[h->nkey], h->fold, h->drow[0].as<uint32_t>(),
                                     h->nkey == 2 ? h->drow[1].as<uint32_t>() : nullptr,
                                     h->drow[h->nkey].as<uint32_t>(), c->stream));
      h->dn = h->didx_n;
      *delta = h->dn;
      return XL_OK;
    }
    if (h->is_minmax) {
      XL_TRY(ensure_drow(h, h->didx_n));
      HIP_TRY(c, k::table16_rows_from_idx(h->table.as<Slot16>(), h->didx.as<uint32_t>(), h->didx_n,
                                          h->kp, h->rel->types[h->nkey], h->fold, h->drow[0].as<uint32_t>(),
                                          h->nkey == 2 ? h->drow[1].as<uint32_t>() : nullptr,
                                          h->drow[h->nkey].as<uint32_t>(), c->stream));
      h->dn = h->didx_n;
      *delta = h->dn;
      return XL_OK;
    }
    // sorted aggregation of this round's candidates
    const int64_t n = h->cn;
    if (n == 0) {
      h->dn = 0;
      *delta = 0;
      return XL_OK;
    }
    const int kbits = h->nkey == 2 ? h->bits0 + h->kp.shift : h->bits0;
    const int kb = (int)key_bytes(h);
    Buf k2, v2, tmp, flag, pos, tot;
    XL_TRY(dalloc(c, (size_t)n * kb, &k2, "sort keys"));
    XL_TRY(dalloc(c, (size_t)n * 4, &v2, "sort values"));
    XL_TRY(dalloc(c, k::radix_temp_bytes(n), &tmp, "sort scratch"));
    int alt = 0;
    if (kb == 4)
      HIP_TRY(c, k::radix_sort_u32(h->ckey.as<uint32_t>(), h->cval.as<uint32_t>(), k2.as<uint32_t>(),
                                   v2.as<uint32_t>(), n, kbits, tmp.p, c->stream, &alt));
    else
      HIP_TRY(c, k::radix_sort_u64(h->ckey.as<u64>(), h->cval.as<uint32_t>(), k2.as<u64>(), v2.as<uint32_t>(),
                                   n, kbits, tmp.p, c->stream, &alt));
    void* sk = alt ? k2.p : h->ckey.p;
    uint32_t* sv = alt ? v2.as<uint32_t>() : h->cval.as<uint32_t>();
    XL_TRY(dalloc(c, (size_t)n * 4, &flag, "segment flags"));
    XL_TRY(dalloc(c, (size_t)n * 4, &pos, "segment ids"));
    XL_TRY(dalloc(c, 8, &tot, "count"));
    tmp.reset();
    XL_TRY(dalloc(c, k::scan_temp_bytes(n), &tmp, "scan scratch"));
    HIP_TRY(c, k::seg_heads(sk, kb, n, flag.as<uint32_t>(), c->stream));
    HIP_TRY(c, k::scan_exclusive_u32(flag.as<uint32_t>(), pos.as<uint32_t>(), n, tot.as<uint32_t>(), tmp.p,
                                     c->stream));
    uint32_t nseg = 0;
    XL_TRY(ctl_read(c, tot.p, 4, &nseg));
    Buf starts;
    XL_TRY(dalloc(c, (size_t)nseg * 4, &starts, "segment starts"));
    HIP_TRY(c, k::seg_starts(flag.as<uint32_t>(), pos.as<uint32_t>(), n, starts.as<uint32_t>(), c->stream));
    XL_TRY(ensure_drow(h, nseg));
    HIP_TRY(c, k::seg_reduce(sk, kb, sv, starts.as<uint32_t>(), nseg, n, h->kp, h->rel->types[h->nkey], h->fold,
                             h->drow[0].as<uint32_t>(), h->nkey == 2 ? h->drow[1].as<uint32_t>() : nullptr,
                             h->drow[h->nkey].as<uint32_t>(), c->stream));
    if (h->ds) {  // seed round of a dense head: the folded rows become the first delta
      HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
      HIP_TRY(c, k::dense_apply_rows(h->drow[0].as<uint32_t>(), h->drow[1].as<uint32_t>(), h->drow[2].as<uint32_t>(),
                                     nseg, h->dmap.as<uint32_t>(), (uint32_t)h->dmap_n, (uint32_t)h->range1,
                                     (uint32_t)h->nrank_d, h->kp,
                                     h->fold, h->rel->types[h->nkey], h->dcur.as<uint32_t>(),
                                     h->dcur_pres.as<uint32_t>(), h->dvals.as<uint32_t>(), h->dpres.as<uint32_t>(),
                                     c->dcounters, c->stream));
      u64 cnt[CNT_N];
      XL_TRY(ctl_read(c, c->dcounters, sizeof(cnt), cnt));
      if (cnt[CNT_FATAL]) return c->fail(XL_DEVICE_ERROR, "key outside the dense domain (internal)");
      h->keys += (int64_t)cnt[CNT_INSERTED];
      if (h->rel->max_rows > 0 && h->keys > h->rel->max_rows)
        return c->fail(XL_CAPACITY_EXCEEDED, "relation " + h->rel->name + " exceeds its max_rows");
      h->dn = nseg;
      h->cn = 0;
      *delta = nseg;
      return XL_OK;
    }
    if (h->keys + (int64_t)nseg > h->cap / 2) XL_TRY(grow(h, h->keys + nseg));
    HIP_TRY(c, hipMemsetAsync(c->dcounters, 0, 8 * CNT_N, c->stream));
    HIP_TRY(c, k::agg_merge(h->table.as<Slot16>(), (u64)h->cap - 1, h->drow[0].as<uint32_t>(),
                            h->nkey == 2 ? h->drow[1].as<uint32_t>() : nullptr, h->drow[h->nkey].as<uint32_t>(),
                            nseg, h->kp, h->rel->types[h->nkey], h->fold, c->dcounters, c->stream));
    u64 cnt[CNT_N];
    XL_TRY(ctl_read(c, c->dcounters, sizeof(cnt), cnt));
    if (cnt[CNT_FATAL]) return c->fail(XL_DEVICE_ERROR, "hash table probe exhausted (internal)");
    h->keys += (int64_t)cnt[CNT_INSERTED];
    if (h->rel->max_rows > 0 && h->keys > h->rel->max_rows)
      return c->fail(XL_CAPACITY_EXCEEDED, "relation " + h->rel->name + " exceeds its max_rows");
    h->dn = nseg;
    h->cn = 0;
    *delta = nseg;
    return XL_OK;
  }

  // Key-column bounds come from the planner's domains (a superset is enough
  // for packing and index ranges); i32 value columns are scanned.
  xl_status set_bounds(HeadRun* h) {
    Relation* r = h->rel;
    if (r->nrows == 0) return XL_OK;
    for (int j = 0; j < h->nkey; ++j) {
      r->lo[j] = (int32_t)h->dom_lo[j];
      r->hi[j] = (int32_t)h->dom_hi[j];
    }
    if (h->nkey < r->arity && r->types[h->nkey] == T_I32 && !h->vbounds) {
      Buf mm;
      XL_TRY(dalloc(c, 8, &mm, "bounds"));
      if (r->nrows <= BOUNDS_ONE_MAX) {
        HIP_TRY(c, k::bounds_one((const int32_t*)r->col[h->nkey], nullptr, r->nrows, mm.as<int32_t>(), c->stream));
      } else {
        HIP_TRY(c, hipMemsetD32Async(mm.as<int32_t>(), INT32_MAX, 1, c->stream));
        HIP_TRY(c, hipMemsetD32Async(mm.as<int32_t>() + 1, INT32_MIN, 1, c->stream));
        HIP_TRY(c, k::minmax_i32((const int32_t*)r->col[h->nkey], r->nrows, mm.as<int32_t>(), c->stream));
      }
      int32_t out[2];
      XL_TRY(ctl_read(c, mm.p, 8, out));
      r->lo[h->nkey] = out[0];
      r->hi[h->nkey] = out[1];
    }
    return XL_OK;
  }

  xl_status materialize(HeadRun* h) {
    XL_TRY(materialize_rows(h));
    return set_bounds(h);
  }

  xl_status materialize_rows(HeadRun* h) {
    Relation* r = h->rel;
    if (h->dense && h->nkey == 1) {  // one bitmap row: the set bits in order
      const int64_t nbits = (h->range0 + 31) / 32 * 32;
      Buf tmp, tot, out;
      XL_TRY(dalloc(c, k::bits_list_temp_bytes(nbits), &tmp, "compaction scratch"));
      XL_TRY(dalloc(c, 8, &tot, "count"));
      XL_TRY(dalloc(c, (size_t)std::max<int64_t>(h->keys, 1) * 4, &out, "relation column"));
      HIP_TRY(c, k::bits_keys(h->bits.as<uint32_t>(), nbits, 1, h->kp.lo[0], 0, 1, false, out.as<uint32_t>(), nullptr,
                              tot.as<uint32_t>(), tmp.p, false, c->stream));
      uint32_t n = 0;
      XL_TRY(ctl_read(c, tot.p, 4, &n));
      if ((int64_t)n != h->keys) return c->fail(XL_DEVICE_ERROR, "bitmap key count mismatch (internal)");
      HIP_TRY(c, k::bits_keys(h->bits.as<uint32_t>(), nbits, 1, h->kp.lo[0], 0, 1, false, out.as<uint32_t>(), nullptr,
                              tot.as<uint32_t>(), tmp.p, true, c->stream));
      h->rows[0].reset();
      relation_free_storage(r);
      r->col[0] = (uint32_t*)out.keep();
      r->nrows = n;
      return XL_OK;
    }
    if (h->dense) {  // every tuple is a set bit: rows in ascending (x, y)
      // off (range0 + 1 words) doubles as the CSR offsets of the finished
      // relation by its first column, kept as a ready index for later strata
      Buf cnt, off, tmp;
      XL_TRY(dalloc(c, (size_t)h->range0 * 4, &cnt, "row counts"));
      XL_TRY(dalloc(c, (size_t)(h->range0 + 1) * 4, &off, "row offsets"));
      XL_TRY(dalloc(c, k::scan_temp_bytes(h->range0), &tmp, "scan scratch"));
      HIP_TRY(c, k::row_popcount(h->bits.as<uint32_t>(), h->range0, h->row_words, cnt.as<uint32_t>(), c->stream));
      HIP_TRY(c, k::scan_exclusive_u32(cnt.as<uint32_t>(), off.as<uint32_t>(), h->range0,
                                       off.as<uint32_t>() + h->range0, tmp.p, c->stream));
      // the receipt's count is the row count; the bitmap's own total is
      // compared on the device (flag read at the end of the run), and the
      // rows are written only up to the allocated count
      const int64_t n = h->keys;
      HIP_TRY(c, k::check_eq(off.as<uint32_t>() + h->range0, (uint32_t)n, c->dcheck, CHECK_BITMAP_ROWS, c->stream));
      h->rows[0].reset();
      h->rows[1].reset();
      Buf out[2];
      for (int j = 0; j < 2; ++j) XL_TRY(dalloc(c, (size_t)std::max<int64_t>(n, 1) * 4, &out[j], "relation column"));
      HIP_TRY(c, k::bits_to_rows(h->bits.as<uint32_t>(), h->range0, h->row_words, off.as<uint32_t>(), h->kp.lo[0],
                                 h->kp.lo[1], out[0].as<uint32_t>(), out[1].as<uint32_t>(), n, c->stream));
      relation_free_storage(r);
      for (int j = 0; j < 2; ++j) r->col[j] = (uint32_t*)out[j].keep();
      r->nrows = n;
      auto ix = std::make_unique<DevIndex>();
      ix->rel = r;
      ix->col = 0;
      ix->probe.off = off.as<uint32_t>();
      ix->probe.ncols = 2;
      for (int j = 0; j < 2; ++j) ix->probe.col[j] = r->col[j];
      ix->probe.key_lo = h->kp.lo[0];
      ix->probe.key_range = (uint32_t)h->range0;
      ix->owned.push_back(std::make_unique<Buf>(c));
      ix->owned.back()->p = off.keep();
      kept.push_back(std::move(ix));
      return XL_OK;
    }
    if (h->dcount) {
      const int64_t n = h->range0 * h->range1;
      Buf tmp, tot;
      XL_TRY(dalloc(c, k::compact_temp_bytes(n), &tmp, "compaction scratch"));
      XL_TRY(dalloc(c, 16, &tot, "count"));
      if (n <= BOUNDS_ONE_MAX) {
        // few slots: the rows go to columns sized for every slot, and their
        // count and the value column's bounds come back in one read
        Buf out[3];
        for (int j = 0; j <= h->nkey; ++j) XL_TRY(dalloc(c, (size_t)std::max<int64_t>(n, 1) * 4, &out[j], "relation column"));
        HIP_TRY(c, k::dcount_rows(h->counts.as<uint32_t>(), n, h->range1, h->kp, out[0].as<uint32_t>(),
                                  h->nkey == 2 ? out[1].as<uint32_t>() : nullptr, out[h->nkey].as<uint32_t>(),
                                  std::max<int64_t>(n, 1), tot.as<uint32_t>(), tmp.p, c->stream));
        const bool i32 = r->types[h->nkey] == T_I32;
        if (i32)
          HIP_TRY(c, k::bounds_one(out[h->nkey].as<int32_t>(), tot.as<uint32_t>(), n, tot.as<int32_t>() + 1,
                                   c->stream));
        int32_t t[3] = {0, 0, 0};
        XL_TRY(ctl_read(c, tot.p, i32 ? 12 : 4, t));
        const uint32_t m = (uint32_t)t[0];
        relation_free_storage(r);
        for (int j = 0; j <= h->nkey; ++j) r->col[j] = (uint32_t*)out[j].keep();
        r->nrows = (int64_t)m;
        h->keys = (int64_t)m;
        if (i32 && m > 0) {
          r->lo[h->nkey] = t[1];
          r->hi[h->nkey] = t[2];
          h->vbounds = true;
        }
        if (r->max_rows > 0 && r->nrows > r->max_rows)
          return c->fail(XL_CAPACITY_EXCEEDED, "relation " + r->name + " exceeds its max_rows");
        return XL_OK;
      }
      HIP_TRY(c, k::dcount_rows(h->counts.as<uint32_t>(), n, h->range1, h->kp, nullptr, nullptr, nullptr, 0,
                                tot.as<uint32_t>(), tmp.p, c->stream));
      uint32_t m = 0;
      XL_TRY(ctl_read(c, tot.p, 4, &m));
      Buf out[3];
      for (int j = 0; j <= h->nkey; ++j) XL_TRY(dalloc(c, (size_t)std::max<uint32_t>(m, 1) * 4, &out[j], "relation column"));
      HIP_TRY(c, k::dcount_rows(h->counts.as<uint32_t>(), n, h->range1, h->kp, out[0].as<uint32_t>(),
                                h->nkey == 2 ? out[1].as<uint32_t>() : nullptr, out[h->nkey].as<uint32_t>(),
                                (int64_t)m, tot.as<uint32_t>(), tmp.p, c->stream));
      relation_free_storage(r);
      for (int j = 0; j <= h->nkey; ++j) r->col[j] = (uint32_t*)out[j].keep();
      r->nrows = (int64_t)m;
      h->keys = (int64_t)m;
      if (r->max_rows > 0 && r->nrows > r->max_rows)
        return c->fail(XL_CAPACITY_EXCEEDED, "relation " + r->name + " exceeds its max_rows");
      return XL_OK;
    }
    if (h->dv) {
      const int64_t n = h->keys;
      const int64_t ns = full_slots(h);
      Buf out[3], tmp, tot;
      for (int j = 0; j <= h->nkey; ++j) XL_TRY(dalloc(c, (size_t)std::max<int64_t>(n, 1) * 4, &out[j], "relation column"));
      XL_TRY(dalloc(c, k::compact_temp_bytes(ns), &tmp, "compaction scratch"));
      XL_TRY(dalloc(c, 8, &tot, "count"));
      HIP_TRY(c, k::dense_rows(h->dvals.as<uint32_t>(), h->dpres.as<uint32_t>(), h->dict.as<uint32_t>(), ns,
                               h->range1, full_nrank(h), h->kp, r->types[h->nkey], h->fold, out[0].as<uint32_t>(),
                               h->nkey == 2 ? out[1].as<uint32_t>() : nullptr, out[h->nkey].as<uint32_t>(),
                               std::max<int64_t>(n, 1), tot.as<uint32_t>(), tmp.p, c->stream));
      uint32_t m = 0;
      XL_TRY(ctl_read(c, tot.p, 4, &m));
      if ((int64_t)m != n) return c->fail(XL_DEVICE_ERROR, "dense value count mismatch (internal)");
      relation_free_storage(r);
      for (int j = 0; j <= h->nkey; ++j) r->col[j] = (uint32_t*)out[j].keep();
      r->nrows = n;
    } else if (h->is_set) {
      relation_free_storage(r);
      for (int j = 0; j < h->nkey; ++j) r->col[j] = (uint32_t*)h->rows[j].keep();
      r->nrows = h->nrows;
    } else {
      Buf out[3];
      const int64_t n = h->keys;
      for (int j = 0; j <= h->nkey; ++j) XL_TRY(dalloc(c, (size_t)std::max<int64_t>(n, 1) * 4, &out[j], "relation column"));
      Buf tmp, tot;
      XL_TRY(dalloc(c, k::compact_temp_bytes(h->cap), &tmp, "compaction scratch"));
      XL_TRY(dalloc(c, 8, &tot, "count"));
      HIP_TRY(c, k::table16_compact(h->table.as<Slot16>(), h->cap, h->kp, r->types[h->nkey], h->fold,
                                    out[0].as<uint32_t>(), h->nkey == 2 ? out[1].as<uint32_t>() : nullptr,
                                    out[h->nkey].as<uint32_t>(), std::max<int64_t>(n, 1), tot.as<uint32_t>(), tmp.p,
                                    c->stream));
      uint32_t m = 0;
      XL_TRY(ctl_read(c, tot.p, 4, &m));
      if ((int64_t)m != n) return c->fail(XL_DEVICE_ERROR, "table compaction count mismatch (internal)");
      relation_free_storage(r);
      for (int j = 0; j <= h->nkey; ++j) r->col[j] = (uint32_t*)out[j].keep();
      r->nrows = n;
    }
    return XL_OK;
  }

  // Indexes over heads of the running stratum describe the relation as it
  // was when they were built; each pass rebuilds them from the current rows.
  // All of a pass's joins with a head of the stratum read the relation as it
  // was when the pass began (Alg. 1: every variant of round k sees S_k), so
  // those indexes are built up front, before any variant adds tuples.
  xl_status snapshot_head_indexes(const std::vector<RulePlan>& plans) {
    indexes.erase(std::remove_if(indexes.begin(), indexes.end(),
                                 [&](const std::unique_ptr<DevIndex>& ix) { return head_of(ix->rel) != nullptr; }),
                  indexes.end());
    for (const RulePlan& p : plans)
      for (const StepPlan& sp : p.steps)
        if (head_of(sp.rel)) {
          IndexProbe probe;
          XL_TRY(get_index(sp.rel, sp.key_col, &probe));
        }
    return XL_OK;
  }

  // ------------------------------------------------------------ strata
  // A triangle-join stratum (see RulePlan::wcoj): count -> scan ->
  // materialize straight into the head's columns, in ascending (X, Y, Z)
  // order; no hash table or bitmap is needed because every (driver row, Z)
  // pair is produced once.
  xl_status run_wcoj(const RulePlan& p) {
    Relation* h = p.head;
    relation_free_storage(h);
    WcojArgs a{};
    IndexProbe ia{};
    XL_TRY(get_index(p.driver, p.tri_a[0], &ia, p.tri_a[1], nullptr, 1));
    XL_TRY(get_index(p.tri_brel, p.tri_b[0], &a.ib, p.tri_b[1], nullptr, 1));
    XL_TRY(get_index(p.tri_crel, p.tri_c[0], &a.ic, p.tri_c[1], nullptr, 1));
    a.ax = ia.col[p.tri_a[0]];
    a.ay = ia.col[p.tri_a[1]];
    a.na = p.driver->nrows;
    a.bz = a.ib.col[p.tri_b[1]];
    a.cz = a.ic.col[p.tri_c[1]];
    a.probe_shorter = c->wcoj_shorter;
    auto finish = [&](int64_t n) -> xl_status {
      h->nrows = n;
      h->lo[0] = p.driver->lo[p.tri_a[0]];
      h->hi[0] = p.driver->hi[p.tri_a[0]];
      h->lo[1] = p.driver->lo[p.tri_a[1]];
      h->hi[1] = p.driver->hi[p.tri_a[1]];
      h->lo[2] = p.tri_brel->lo[p.tri_b[1]];
      h->hi[2] = p.tri_brel->hi[p.tri_b[1]];
      record(n);
      st->new_tuples_total += n;
      return XL_OK;
    };
    if (a.na == 0 || p.tri_brel->nrows == 0 || p.tri_crel->nrows == 0) return finish(0);
    Buf work, flags, flag_pos, crow, cw, cofs, tmp, tot;
    XL_TRY(dalloc(c, (size_t)a.na * 4, &work, "triangle work"));
    XL_TRY(dalloc(c, (size_t)a.na * 4, &flags, "triangle row flags"));
    XL_TRY(dalloc(c, (size_t)a.na * 4, &flag_pos, "triangle row positions"));
    XL_TRY(dalloc(c, std::max(k::scan_temp_bytes(a.na), k::scan_temp_bytes(a.na + 1)), &tmp, "scan scratch"));
    XL_TRY(dalloc(c, 16, &tot, "count"));
    a.work = work.as<uint32_t>();
    HIP_TRY(c, k::wcoj_work(a, c->stream));
    // flags and positions in separate arrays: the scan then takes its
    // one-launch form (it reads other tiles' flags)
    HIP_TRY(c, k::nonzero_flags(work.as<uint32_t>(), a.na, flags.as<uint32_t>(), c->stream));
    HIP_TRY(c, k::scan_exclusive_u32(flags.as<uint32_t>(), flag_pos.as<uint32_t>(), a.na, tot.as<uint32_t>(), tmp.p,
                                     c->stream));
    uint32_t nz = 0;
    XL_TRY(ctl_read(c, tot.p, 4, &nz));
    if (nz == 0) return finish(0);
    XL_TRY(dalloc(c, (size_t)nz * 4, &crow, "triangle rows"));
    XL_TRY(dalloc(c, (size_t)(nz + 1) * 8, &cw, "triangle row work"));
    XL_TRY(dalloc(c, (size_t)(nz + 1) * 8, &cofs, "triangle row offsets"));
    HIP_TRY(c, k::wcoj_compact(work.as<uint32_t>(), flag_pos.as<uint32_t>(), a.na, crow.as<uint32_t>(),
                               cw.as<unsigned long long>(), c->stream));
    XL_TRY(dalloc(c, k::scan_temp_bytes(nz), &tmp, "scan scratch"));
    HIP_TRY(c, k::scan_exclusive_u64(cw.as<u64>(), cofs.as<u64>(), nz, cofs.as<u64>() + nz, tmp.p, c->stream));
    u64 items = 0;
    XL_TRY(ctl_read(c, cofs.as<u64>() + nz, 8, &items));
    if (items >= ((u64)1 << 40)) return c->fail(XL_UNSUPPORTED, "triangle join with more than 2^40 probes");
    a.crow = crow.as<uint32_t>();
    a.cofs = cofs.as<unsigned long long>();
    a.nz = nz;
    a.items = items;
    const u64 nchunks = (items + k::WC_CHUNK - 1) / k::WC_CHUNK;
    Buf ccnt, coff, tmp2;
    XL_TRY(dalloc(c, (size_t)nchunks * 4, &ccnt, "chunk counts"));
    XL_TRY(dalloc(c, (size_t)nchunks * 4, &coff, "chunk offsets"));
    XL_TRY(dalloc(c, k::scan_temp_bytes((int64_t)nchunks), &tmp2, "scan scratch"));
    a.chunk_cnt = ccnt.as<uint32_t>();
    float ms_total = 0;
    auto timed = [&](bool mat) -> xl_status {
      if (c->profile) HIP_TRY(c, hipEventRecord(ev[0], c->stream));
      HIP_TRY(c, k::wcoj_probe(a, mat, c->stream));
      if (c->profile) {
        HIP_TRY(c, hipEventRecord(ev[1], c->stream));
        HIP_TRY(c, hipEventSynchronize(ev[1]));
        float ms = 0;
        HIP_TRY(c, hipEventElapsedTime(&ms, ev[0], ev[1]));
        ms_total += ms;
      }
      return XL_OK;
    };
    XL_TRY(timed(false));
    HIP_TRY(c, k::scan_exclusive_u32(ccnt.as<uint32_t>(), coff.as<uint32_t>(), (int64_t)nchunks, tot.as<uint32_t>(),
                                     tmp2.p, c->stream));
    uint32_t n = 0;
    XL_TRY(ctl_read(c, tot.p, 4, &n));
    if (h->max_rows > 0 && (int64_t)n > h->max_rows)
      return c->fail(XL_CAPACITY_EXCEEDED, "relation " + h->name + " exceeds its max_rows " +
                                               std::to_string(h->max_rows));
    Buf out[3];
    for (int j = 0; j < 3; ++j) XL_TRY(dalloc(c, (size_t)std::max<uint32_t>(n, 1) * 4, &out[j], "relation column"));
    a.chunk_off = coff.as<uint32_t>();
    a.out0 = out[0].as<uint32_t>();
    a.out1 = out[1].as<uint32_t>();
    a.out2 = out[2].as<uint32_t>();
    if (n) XL_TRY(timed(true));
    cands += (int64_t)items;
    if (c->profile) {
      st->wcoj_ms += ms_total;
      st->wcoj_launches += n ? 2 : 1;
      st->wcoj_candidates += (int64_t)items;
      st->wcoj_new += n;
    }
    for (int j = 0; j < 3; ++j) h->col[j] = (uint32_t*)out[j].keep();
    return finish(n);
  }

  xl_status run_stratum(Stratum& s, int64_t max_iterations) {
    if (s.full.size() == 1 && s.full[0].wcoj) {
      heads.clear();
      return run_wcoj(s.full[0]);
    }
    heads.clear();
    // rows the heads keep from before the run (set, min and max heads resume;
    // count, sum and logsumexp heads are recomputed from empty)
    int64_t rows_before = 0;
    for (Relation* h : s.heads) {
      const Agg a = prog->head_agg(h);
      if (a == Agg::NONE || a == Agg::MIN || a == Agg::MAX) rows_before += h->nrows;
    }
    XL_TRY(setup_heads(s));
    for (auto& h : heads) begin_round(h.get());
    XL_TRY(snapshot_head_indexes(s.full));
    // A stratum that runs as one resident frontier launch builds that
    // launch's indexes (inputs only) while its seed round runs: the host's
    // launches then overlap the seed kernel instead of following its count
    // read.
    struct ClearHook {
      std::function<xl_status()>& f;
      ~ClearHook() { f = nullptr; }
    } clear_hook{before_count_read};
    if (s.recursive && heads.size() == 1 && heads[0]->resident && s.variants.size() == 1 &&
        s.variants[0].driver_delta && head_of(s.variants[0].head) == heads[0].get())
      before_count_read = [this, &s]() {
        FrontierArgs f{};
        return frontier_args(s.variants[0], heads[0].get(), f);
      };
    for (RulePlan& p : s.full) XL_TRY(eval_plan(p));
    before_count_read = nullptr;
    int64_t total = 0;
    for (auto& h : heads) {
      int64_t d = 0;
      XL_TRY(finish_round(h.get(), &d));
      total += d;
      st->new_tuples_total += d;
    }
    const int32_t seed_record = st->rounds_recorded;
    record(total);
    if (s.recursive && total > 0 && batched_tiles(s)) {
      XL_TRY(run_tiles_batched(s.variants[0], heads[0].get(), max_iterations));
      total = 0;
    }
    if (s.recursive && total > 0 && batched_pull(s)) {
      XL_TRY(run_pull_batched(s.variants[0], heads[0].get(), max_iterations));
      total = 0;
    }
    if (s.recursive && total > 0 && batched_gather(s)) {
      XL_TRY(run_gather_batched(s.variants[0], heads[0].get(), max_iterations));
      total = 0;
    }
    if (s.recursive && total > 0 && batched_sets(s)) {
      XL_TRY(run_sets_batched(s, max_iterations));
      total = 0;
    }
    if (s.recursive && total > 0 && batched_values(s)) {
      XL_TRY(run_values_batched(s, heads[0].get(), max_iterations));
      total = 0;
    }
    if (s.recursive && total > 0 && resident_frontier(s)) {
      if (max_iterations == 0)
        return c->fail(XL_CONVERGENCE_FAILURE, "iteration cap 0 reached before the fixpoint");
      XL_TRY(run_frontier_resident(s.variants[0], heads[0].get(), max_iterations));
      total = 0;
    }
    if (s.recursive) {
      int64_t pass = 0;
      while (total > 0) {
        if (pass >= max_iterations)
          return c->fail(XL_CONVERGENCE_FAILURE, "iteration cap " + std::to_string(max_iterations) +
                                                     " reached before the fixpoint");
        ++pass;
        st->iterations++;
        for (auto& h : heads) begin_round(h.get());
        XL_TRY(snapshot_head_indexes(s.variants));
        for (RulePlan& p : s.variants) XL_TRY(eval_plan(p));
        total = 0;
        for (auto& h : heads) {
          int64_t d = 0;
          XL_TRY(finish_round(h.get(), &d));
          total += d;
          st->new_tuples_total += d;
        }
        record(total);
      }
    }
    // indexes over this stratum's heads saw unfinished relations; the rest
    // stay valid (a relation is final once its stratum ends)
    for (auto& h : heads)
      indexes.erase(std::remove_if(indexes.begin(), indexes.end(),
                                   [&](const std::unique_ptr<DevIndex>& ix) { return ix->rel == h->rel; }),
                    indexes.end());
    kept.clear();
    for (auto& h : heads) XL_TRY(materialize(h.get()));
    if (!s.recursive && seed_record < XL_STATS_ROUNDS) {
      // a non-recursive stratum records the rows it produced; aggregate heads
      // built from sorted segments or index degrees only have them now
      int64_t produced = -rows_before;
      for (auto& h : heads) produced += h->rel->nrows;
      st->new_tuples_total += produced - st->delta_rows[seed_record];
      st->delta_rows[seed_record] = produced;
    }
    for (auto& ix : kept) indexes.push_back(std::move(ix));
    kept.clear();
    heads.clear();
    return XL_OK;
  }
};

}  // namespace

xl_status run_program(Program* p, int64_t max_iterations, xl_fixpoint_stats* st) {
  Context* c = p->ctx;
  memset(st, 0, sizeof(*st));
  if (c->device < 0) return c->fail(XL_INVALID_ARGUMENT, "planning-only context cannot run programs");
  if (max_iterations < 0) return c->fail(XL_INVALID_ARGUMENT, "negative iteration cap");
  c->arena.reset_peak();
  c->runs++;
  const int64_t ctl0 = c->control_bytes;
  {
    const xl_status s0 = resolve_wide_constants(p);
    if (s0 != XL_OK) {
      st->status = s0;
      return s0;
    }
  }
  hipEvent_t e0, e1;
  HIP_TRY(c, hipEventCreate(&e0));
  HIP_TRY(c, hipEventCreate(&e1));
  HIP_TRY(c, hipEventRecord(e0, c->stream));
  HIP_TRY(c, hipMemsetAsync(c->dcheck, 0, 8, c->stream));
  xl_status s = XL_OK;
  {
    Runner run{c, p, st};
    if (c->profile) {
      HIP_TRY(c, hipEventCreate(&run.ev[0]));
      HIP_TRY(c, hipEventCreate(&run.ev[1]));
    }
    for (Stratum& str : p->strata) {
      s = run.run_stratum(str, max_iterations);
      if (s != XL_OK) break;
    }
    st->candidates_total = run.cands;
  }
  // the consistency flags ride on the run's final synchronization: the copy
  // into the control block's last word is complete once e1 is
  unsigned long long* check_host = (unsigned long long*)((char*)c->pinned + CTL_CHECK_OFFSET);
  *check_host = 0;
  (void)hipMemcpyAsync(check_host, c->dcheck, 8, hipMemcpyDeviceToHost, c->stream);
  (void)hipEventRecord(e1, c->stream);
  (void)hipEventSynchronize(e1);
  if (s == XL_OK && *check_host) {
    const unsigned long long f = *check_host;
    s = c->fail(XL_DEVICE_ERROR, std::string("internal consistency check failed:") +
                                     (f & CHECK_BITMAP_ROWS ? " bitmap row count" : "") +
                                     (f & CHECK_COUNT_DOMAIN ? " count key outside the head domain" : ""));
  }
  float ms = 0;
  (void)hipEventElapsedTime(&ms, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  st->ms_total = ms;
  st->strata = (int32_t)p->strata.size();
  for (auto& h : p->heads) st->derived_tuples += h.rel->nrows;
  st->peak_workspace_bytes = (int64_t)c->arena.peak();
  st->control_bytes_read = c->control_bytes - ctl0;
  st->status = s;
  return s;
}

}  // namespace xlh
