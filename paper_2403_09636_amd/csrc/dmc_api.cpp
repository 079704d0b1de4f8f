// Host side of the DMC C ABI: configuration and argument validation,
// workspace layout, per-layer state and kernel launches.
//
// Every validation runs before the first HIP call of an entry point, so an
// invalid request returns its status without touching the device (and can
// be exercised on a machine with no GPU).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <algorithm>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/dmc.h"
#include "dmc_internal.h"

using dmc::align_up;

struct dmc_cache {
  dmc_cache_config cfg;
  dmc::Layout lay;
  char *ws;
  size_t ws_bytes;
  int device;
  int cu_count;
};

namespace {

thread_local std::string g_err;

dmc_status fail(dmc_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

dmc_status hip_fail(hipError_t e, const char *what) {
  return fail(DMC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }
int ilog2(int64_t x) {
  int r = 0;
  while ((int64_t(1) << r) < x) ++r;
  return r;
}
bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#ifndef DMC_DECODE_WG_PER_CU
#define DMC_DECODE_WG_PER_CU 2
#endif
// Persistent decode grid, counted in workgroups of 4 waves per compute unit
// (the vector-ALU launch packs them into 8-wave workgroups for bf16 caches
// with up to two query heads per kv head), and the largest number of waves a
// decode launch uses.
constexpr int kDecodeWgPerCu = DMC_DECODE_WG_PER_CU;
constexpr int64_t kMaxDecodeWaves = 8192;
constexpr size_t kMaxDecodeLds = 64 * 1024;
constexpr size_t kMaxLdsPerWorkgroup = 160 * 1024;   // gfx950

int elem_bytes(const dmc_cache_config &c) { return c.dtype == DMC_FP32 ? 4 : 2; }

// Units per entry of the decode kernel's slot-space table in LDS: 1 (every
// unit's offset) when that table fits beside the kernel's static LDS, else the
// smallest power of two that makes it fit (exact caches; windowed ones need
// 1); 0 if none up to kMaxSlotGroup does.
int slot_group_for(const dmc_cache_config &c) {
  const int64_t units = int64_t(c.batch) * c.num_kv_heads;
  const int G = c.num_q_heads / c.num_kv_heads;
  const bool v_trans = c.dtype == DMC_BF16 && G >= 4 && c.page_size == 32;
  // windowed caches decode with the full table only
  const int gmax = c.window > 0 ? 1 : dmc::kMaxSlotGroup;
  for (int g = 1; g <= gmax; g <<= 1) {
    const int entries = static_cast<int>((units + g - 1) / g + 1);
    const size_t dyn = dmc::decode_lds_bytes(entries, G, c.head_dim, c.window > 0);
    if (dyn <= kMaxDecodeLds &&
        dyn + dmc::decode_static_lds_bytes(c.head_dim, v_trans) <= kMaxLdsPerWorkgroup)
      return g;
  }
  return 0;
}

dmc_status validate_config(const dmc_cache_config *c) {
  if (!c) return fail(DMC_ERR_INVALID_ARG, "config is NULL");
  if (c->num_layers < 1 || c->batch < 1 || c->num_kv_heads < 1 || c->num_q_heads < 1)
    return fail(DMC_ERR_INVALID_ARG, "layers, batch and head counts must be >= 1");
  if (c->num_q_heads % c->num_kv_heads != 0)
    return fail(DMC_ERR_INVALID_ARG, "num_q_heads (%d) must be a multiple of num_kv_heads (%d)",
                c->num_q_heads, c->num_kv_heads);
  const int G = c->num_q_heads / c->num_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(DMC_ERR_UNSUPPORTED, "query group size %d not in {1,2,4,8}", G);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(DMC_ERR_UNSUPPORTED, "head_dim %d not in {64,128}", c->head_dim);
  if (c->dtype != DMC_BF16 && c->dtype != DMC_FP32)
    return fail(DMC_ERR_INVALID_ARG, "unknown dtype %d", c->dtype);
  if (!pow2(c->page_size) || c->page_size < 8 || c->page_size > 65536)
    return fail(DMC_ERR_UNSUPPORTED, "page_size %d must be a power of two in [8,65536]",
                c->page_size);
  if (c->max_slots_per_seq < 1)
    return fail(DMC_ERR_INVALID_ARG, "max_slots_per_seq must be >= 1");
  if (c->num_pages < 1 || c->num_pages >= (int64_t(1) << 31))
    return fail(DMC_ERR_INVALID_ARG, "num_pages %lld outside [1, 2^31)",
                static_cast<long long>(c->num_pages));
  if (!std::isfinite(c->decision_bias)) return fail(DMC_ERR_INVALID_ARG, "decision_bias not finite");
  if (c->omega_src != DMC_OMEGA_LEAD_QHEAD && c->omega_src != DMC_OMEGA_GROUP_MEAN &&
      c->omega_src != DMC_OMEGA_UNIFORM)
    return fail(DMC_ERR_INVALID_ARG, "unknown omega_src %d", c->omega_src);
  if (c->decision_src != DMC_DECISION_PER_HEAD && c->decision_src != DMC_DECISION_SHARED_LAYER)
    return fail(DMC_ERR_INVALID_ARG, "unknown decision_src %d", c->decision_src);
  if (c->window < 0) return fail(DMC_ERR_INVALID_ARG, "window must be >= 0");
  if (c->window > dmc::kMaxWindow)
    return fail(DMC_ERR_UNSUPPORTED, "window %d exceeds %d", c->window, dmc::kMaxWindow);
  if (c->split_tile < 0) return fail(DMC_ERR_INVALID_ARG, "split_tile must be >= 0");
  if (c->max_prompt_len < 0 || c->max_prompt_len > c->max_slots_per_seq)
    return fail(DMC_ERR_INVALID_ARG, "max_prompt_len must be in [0, max_slots_per_seq]");
  const int64_t units = int64_t(c->batch) * c->num_kv_heads;
  if (units > (int64_t(1) << 20)) return fail(DMC_ERR_UNSUPPORTED, "too many units per layer");
  if (slot_group_for(*c) == 0)
    return fail(DMC_ERR_UNSUPPORTED,
                "batch * num_kv_heads = %lld units exceed the decode kernel's LDS slot-space table "
                "(%s)", static_cast<long long>(units),
                c->window > 0 ? "a windowed cache keeps one entry per unit"
                              : "even at 64 units per entry");
  return DMC_OK;
}

dmc::Layout make_layout(const dmc_cache_config &c) {
  dmc::Layout L{};
  const int es = elem_bytes(c);
  L.units = c.batch * c.num_kv_heads;
  L.group = c.num_q_heads / c.num_kv_heads;
  L.maxpages = static_cast<int32_t>((int64_t(c.max_slots_per_seq) + c.page_size - 1) / c.page_size);
  L.split_tile = c.split_tile;
  {
    // ranges <= max(waves, ceil(S / split_tile)) with S <= U * max_slots; one
    // record per (range, unit) piece is indexed range + unit.
    const int64_t S = int64_t(L.units) * (c.max_slots_per_seq + dmc::kDecodeUnitOverhead);
    int64_t ranges = kMaxDecodeWaves;
    if (c.split_tile > 0) ranges = std::max<int64_t>(ranges, (S + c.split_tile - 1) / c.split_tile);
    L.max_records = ranges + L.units + 1;
  }
  L.max_prompt = c.max_prompt_len > 0 ? c.max_prompt_len : c.max_slots_per_seq;
  L.prompt_chunks = (L.max_prompt + 63) / 64;
  L.carry_blocks = (L.max_prompt + 31) / 32;
  L.window = c.window;
  L.slot_group = slot_group_for(c);
  L.page_bytes = int64_t(2) * c.page_size * c.head_dim * es;
  // Grouped-query caches decode on matrix cores with value pages transposed.
  L.v_trans = c.dtype == DMC_BF16 && L.group >= 4 && c.page_size == 32;
  const size_t U = size_t(L.units), NL = size_t(c.num_layers);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes, 256);
    return at;
  };
  L.pool = take(size_t(c.num_pages) * size_t(L.page_bytes));
  L.ptab = take(NL * U * size_t(L.maxpages) * 4);
  L.lens = take(2 * NL * U * 4);
  L.z = take(NL * U * 4);
  L.ctrl = take(sizeof(dmc::Control));
  L.meta = take(U * 2 * 4);
  L.partials = take(size_t(L.max_records) * L.group * (c.head_dim + 4) * 4);
  L.pf_alpha = take(U * size_t(L.max_prompt));
  L.pf_omega = take(U * size_t(L.max_prompt) * 4);
  L.pf_count = take(U * size_t(L.prompt_chunks) * 4);
  L.pf_mask = take(U * size_t(L.prompt_chunks) * 8);
  L.pf_pagebase = take(U * 4);
  L.pf_carry = take(U * size_t(L.carry_blocks) * dmc::carry_stride(c.head_dim) * 4);
  L.win = take(NL * U * size_t(L.window) * 2 * c.head_dim * es);
  L.win_omega = take(NL * U * size_t(L.window) * 4);
  L.win_len = take(L.window > 0 ? NL * U * 4 : 0);
  L.total = off;
  return L;
}

// Runs the enqueue on the cache's device, restoring the caller's afterwards.
struct DeviceGuard {
  int prev = -1;
  bool ok = true;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) {
      ok = false;
      return;
    }
    if (prev != dev && hipSetDevice(dev) != hipSuccess) ok = false;
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

template <typename T>
T *at(const dmc_cache *c, size_t off) {
  return reinterpret_cast<T *>(c->ws + off);
}

// Lengths of one layer: buffer 0 holds the current slot counts (read by every
// kernel); buffer 1 receives the post-step counts of a decode step, which the
// step's combine launch copies back into buffer 0.  A decode call therefore
// always uses the same pair, and a captured call replays correctly.
int32_t *lens_of(const dmc_cache *c, int layer, int which) {
  return at<int32_t>(c, c->lay.lens) + (size_t(which) * c->cfg.num_layers + layer) * c->lay.units;
}

// Token-window ring of one layer (all null when the cache has no window).
dmc::WindowState window_of(const dmc_cache *c, int layer) {
  dmc::WindowState w{};
  const dmc::Layout &L = c->lay;
  w.window = L.window;
  if (L.window > 0) {
    const size_t units = size_t(L.units) * L.window;
    w.ring = c->ws + L.win + size_t(layer) * units * 2 * c->cfg.head_dim * elem_bytes(c->cfg);
    w.omega = at<float>(c, L.win_omega) + size_t(layer) * units;
    w.seg_len = at<int32_t>(c, L.win_len) + size_t(layer) * L.units;
  }
  return w;
}

dmc_status check_layer(const dmc_cache *c, int32_t layer) {
  if (!c) return fail(DMC_ERR_INVALID_ARG, "cache is NULL");
  if (layer < 0 || layer >= c->cfg.num_layers)
    return fail(DMC_ERR_INVALID_ARG, "layer %d outside [0, %d)", layer, c->cfg.num_layers);
  return DMC_OK;
}

dmc_status enqueue_reset(dmc_cache *c, hipStream_t s) {
  const size_t U = c->lay.units, NL = c->cfg.num_layers;
  hipError_t e;
  if ((e = dmc::launch_fill_i32(at<int32_t>(c, c->lay.lens), 0, 2 * NL * U, s)) != hipSuccess)
    return hip_fail(e, "reset lengths");
  if ((e = dmc::launch_fill_i32(at<int32_t>(c, c->lay.z), 0, NL * U, s)) != hipSuccess)
    return hip_fail(e, "reset z");
  if ((e = dmc::launch_fill_i32(at<int32_t>(c, c->lay.ptab), -1, NL * U * c->lay.maxpages, s)) !=
      hipSuccess)
    return hip_fail(e, "reset page table");
  if ((e = dmc::launch_fill_u8(c->ws + c->lay.ctrl, sizeof(dmc::Control), s)) != hipSuccess)
    return hip_fail(e, "reset control block");
  if ((e = dmc::launch_fill_i32(at<int32_t>(c, c->lay.meta), 0, 2 * U, s)) != hipSuccess)
    return hip_fail(e, "reset tile table");
  if (c->lay.window > 0 &&
      (e = dmc::launch_fill_i32(at<int32_t>(c, c->lay.win_len), 0, NL * U, s)) != hipSuccess)
    return hip_fail(e, "reset window lengths");
  return DMC_OK;
}

}  // namespace

extern "C" {

const char *dmc_last_error(void) { return g_err.c_str(); }

size_t dmc_cache_workspace_bytes(const dmc_cache_config *cfg) {
  if (validate_config(cfg) != DMC_OK) return 0;
  return make_layout(*cfg).total;
}

dmc_status dmc_cache_alloc(const dmc_cache_config *cfg, void *workspace, size_t bytes,
                           dmc_stream_t stream, dmc_cache **out) {
  if (!out) return fail(DMC_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  dmc_status st = validate_config(cfg);
  if (st != DMC_OK) return st;
  if (!workspace) return fail(DMC_ERR_INVALID_ARG, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(workspace) & 255u)
    return fail(DMC_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  const dmc::Layout lay = make_layout(*cfg);
  if (bytes < lay.total)
    return fail(DMC_ERR_INVALID_ARG, "workspace has %zu bytes, needs %zu", bytes, lay.total);
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
  dmc_cache *c = new (std::nothrow) dmc_cache();
  if (!c) return fail(DMC_ERR_INVALID_ARG, "out of host memory");
  c->cfg = *cfg;
  c->lay = lay;
  c->ws = static_cast<char *>(workspace);
  c->ws_bytes = bytes;
  c->device = dev;
  c->cu_count = cus > 0 ? cus : 256;
  // Set-up of dmc_decode_step_static: the device address of the library's
  // static scratch on this (current) device, resolved once per device.
  void *scratch = nullptr;
  e = dmc::static_scratch(&scratch);
  if (e != hipSuccess) {
    delete c;
    return hip_fail(e, "static scratch address");
  }
  st = enqueue_reset(c, static_cast<hipStream_t>(stream));
  if (st != DMC_OK) {
    delete c;
    return st;
  }
  *out = c;
  return DMC_OK;
}

dmc_status dmc_cache_free(dmc_cache *cache) {
  if (!cache) return fail(DMC_ERR_INVALID_ARG, "cache is NULL");
  delete cache;
  return DMC_OK;
}

dmc_status dmc_cache_reset(dmc_cache *cache, dmc_stream_t stream) {
  if (!cache) return fail(DMC_ERR_INVALID_ARG, "cache is NULL");
  DeviceGuard g(cache->device);
  if (!g.ok) return fail(DMC_ERR_HIP, "cannot select the cache's device");
  return enqueue_reset(cache, static_cast<hipStream_t>(stream));
}

namespace {

// Persistent decode grid of a cache: workgroups of 4 waves, kDecodeWgPerCu per
// compute unit (the matrix-core launch halves it when its LDS ring allows one;
// the vector-ALU launch may pack the same waves into larger workgroups).
int decode_grid(const dmc_cache *cache) {
  return static_cast<int>(
      std::min<int64_t>(int64_t(cache->cu_count) * kDecodeWgPerCu, kMaxDecodeWaves / 4));
}

// Shared checks and parameter set-up of the two decode entry points; the
// split-K records (partials, meta) are filled in by the caller.
dmc_status decode_params(dmc_cache *cache, int32_t layer, const void *q, const void *k,
                         const void *v, void *out, int32_t *slot_index, dmc::DecodeParams *out_p) {
  dmc_status st = check_layer(cache, layer);
  if (st != DMC_OK) return st;
  if (!q || !k || !v || !out) return fail(DMC_ERR_INVALID_ARG, "q, k, v and out must be non-NULL");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(out))
    return fail(DMC_ERR_INVALID_ARG, "q, k, v and out must be 16-byte aligned");
  const dmc_cache_config &c = cache->cfg;
  const dmc::Layout &L = cache->lay;
  dmc::DecodeParams &p = *out_p;
  p = dmc::DecodeParams{};
  p.pool = cache->ws + L.pool;
  p.page_bytes = L.page_bytes;
  p.num_pages = c.num_pages;
  p.ptab = at<int32_t>(cache, L.ptab) + size_t(layer) * L.units * L.maxpages;
  p.len_in = lens_of(cache, layer, 0);
  p.len_out = lens_of(cache, layer, 1);
  p.z = at<float>(cache, L.z) + size_t(layer) * L.units;
  p.ctrl = at<dmc::Control>(cache, L.ctrl);
  p.q = q;
  p.k = k;
  p.v = v;
  p.out = out;
  p.slot_index = slot_index;
  p.win = window_of(cache, layer);
  p.c = c.decision_bias;
  p.scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(double(c.head_dim)));
  p.units = L.units;
  p.hkv = c.num_kv_heads;
  p.hq = c.num_q_heads;
  p.maxpages = L.maxpages;
  p.max_slots = c.max_slots_per_seq;
  p.log2p = ilog2(c.page_size);
  p.split_tile = L.split_tile;
  p.omega_src = c.omega_src;
  p.decision_src = c.decision_src;
  p.slot_group = L.slot_group;
  return DMC_OK;
}

dmc_status decode_launch(dmc_cache *cache, const dmc::DecodeParams &p, dmc_stream_t stream) {
  hipError_t e = dmc::launch_decode(elem_bytes(cache->cfg), cache->cfg.head_dim, cache->lay.group,
                                    cache->lay.v_trans, p, decode_grid(cache),
                                    static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "decode launch");
  return DMC_OK;
}

// Bytes of split-K records one decode launch of this cache can use: the
// per-unit table (first record, count) and one record of G x (d + 4) fp32 per
// (range, unit) piece, indexed range + unit.  Ranges are at most the launch's
// waves, or ceil(S / split_tile) with S <= units * (max_slots_per_seq + the
// decode kernels' virtual positions per unit).
size_t decode_records_bytes(const dmc_cache *cache, size_t *meta_bytes) {
  const dmc::Layout &L = cache->lay;
  int64_t ranges = int64_t(decode_grid(cache)) * 4;
  if (L.split_tile > 0) {
    const int64_t S = int64_t(L.units) * (cache->cfg.max_slots_per_seq + dmc::kDecodeUnitOverhead);
    ranges = std::max<int64_t>(ranges, (S + L.split_tile - 1) / L.split_tile);
  }
  *meta_bytes = align_up(size_t(L.units) * 2 * 4, 256);
  return *meta_bytes + size_t(ranges + L.units) * L.group * (cache->cfg.head_dim + 4) * 4;
}

}  // namespace

dmc_status dmc_decode_step(dmc_cache *cache, int32_t layer, const void *q, const void *k,
                           const void *v, void *out, int32_t *slot_index, dmc_stream_t stream) {
  dmc::DecodeParams p;
  dmc_status st = decode_params(cache, layer, q, k, v, out, slot_index, &p);
  if (st != DMC_OK) return st;
  p.partials = at<float>(cache, cache->lay.partials);
  p.meta = at<int32_t>(cache, cache->lay.meta);
  DeviceGuard g(cache->device);
  if (!g.ok) return fail(DMC_ERR_HIP, "cannot select the cache's device");
  return decode_launch(cache, p, stream);
}

dmc_status dmc_decode_step_static(dmc_cache *cache, int32_t layer, const void *q, const void *k,
                                  const void *v, void *out, int32_t *slot_index,
                                  dmc_stream_t stream) {
  dmc::DecodeParams p;
  dmc_status st = decode_params(cache, layer, q, k, v, out, slot_index, &p);
  if (st != DMC_OK) return st;
  size_t meta_bytes = 0;
  const size_t need = decode_records_bytes(cache, &meta_bytes);
  if (need > dmc::kStaticScratchBytes)
    return fail(DMC_ERR_UNSUPPORTED,
                "decode records of this cache need %zu bytes, more than the %zu-byte static "
                "scratch of dmc_decode_step_static (use dmc_decode_step)",
                need, dmc::kStaticScratchBytes);
  DeviceGuard g(cache->device);
  if (!g.ok) return fail(DMC_ERR_HIP, "cannot select the cache's device");
  char *scratch = nullptr;
  hipError_t e = dmc::static_scratch(reinterpret_cast<void **>(&scratch));
  if (e != hipSuccess) return hip_fail(e, "static scratch address");
  p.meta = reinterpret_cast<int32_t *>(scratch);
  p.partials = reinterpret_cast<float *>(scratch + meta_bytes);
  return decode_launch(cache, p, stream);
}

namespace {

// Shared argument checks and parameter set-up of the two prompt entry points.
dmc_status prefill_params(dmc_cache *cache, int32_t layer, const void *k, const int64_t k_strides[3],
                          const void *v, const int64_t v_strides[3], const void *q,
                          const int64_t q_strides[3], int32_t n, const int32_t *prompt_lens,
                          int32_t *slot_index, bool full_q, dmc::PrefillParams *out) {
  dmc_status st = check_layer(cache, layer);
  if (st != DMC_OK) return st;
  const dmc_cache_config &c = cache->cfg;
  const dmc::Layout &L = cache->lay;
  if (n < 0 || n > L.max_prompt)
    return fail(DMC_ERR_INVALID_ARG, "prompt length %d outside [0, %d]", n, L.max_prompt);
  if (n > 0) {
    if (!k || !v || !q) return fail(DMC_ERR_INVALID_ARG, "k, v and q must be non-NULL");
    if (!k_strides || !v_strides || !q_strides)
      return fail(DMC_ERR_INVALID_ARG, "stride arrays must be non-NULL");
    if (!aligned16(k) || !aligned16(v))
      return fail(DMC_ERR_INVALID_ARG, "k and v must be 16-byte aligned");
    if (full_q && !aligned16(q)) return fail(DMC_ERR_INVALID_ARG, "q must be 16-byte aligned");
    for (int i = 0; i < 3; ++i) {
      if (k_strides[i] < 0 || v_strides[i] < 0 || q_strides[i] < 0)
        return fail(DMC_ERR_INVALID_ARG, "strides must be non-negative");
      if (k_strides[i] % 8 || v_strides[i] % 8)
        return fail(DMC_ERR_INVALID_ARG, "k and v strides must be multiples of 8 elements");
      if (full_q && q_strides[i] % 8)
        return fail(DMC_ERR_INVALID_ARG, "q strides must be multiples of 8 elements");
    }
    // the compaction addresses up to 64 consecutive tokens from one base with
    // 32-bit offsets
    const int64_t es = c.dtype == DMC_FP32 ? 4 : 2, lim = int64_t(1) << 25;
    if (k_strides[1] * es >= lim || v_strides[1] * es >= lim || q_strides[1] * es >= lim)
      return fail(DMC_ERR_UNSUPPORTED, "k, v and q token strides must be below 32 MiB");
  }
  dmc::PrefillParams &p = *out;
  p = dmc::PrefillParams{};
  p.pool = cache->ws + L.pool;
  p.page_bytes = L.page_bytes;
  p.num_pages = c.num_pages;
  p.ptab = at<int32_t>(cache, L.ptab) + size_t(layer) * L.units * L.maxpages;
  p.len = lens_of(cache, layer, 0);
  p.z = at<float>(cache, L.z) + size_t(layer) * L.units;
  p.ctrl = at<dmc::Control>(cache, L.ctrl);
  p.k = k;
  p.v = v;
  p.q = q;
  for (int i = 0; i < 3; ++i) {
    p.ks[i] = n > 0 ? k_strides[i] : 0;
    p.vs[i] = n > 0 ? v_strides[i] : 0;
    p.qs[i] = n > 0 ? q_strides[i] : 0;
  }
  p.prompt_lens = prompt_lens;
  p.slot_index = slot_index;
  p.alpha = at<uint8_t>(cache, L.pf_alpha);
  p.omega = at<float>(cache, L.pf_omega);
  p.count = at<int32_t>(cache, L.pf_count);
  p.mask = at<uint64_t>(cache, L.pf_mask);
  p.page_base = at<int32_t>(cache, L.pf_pagebase);
  p.carry = nullptr;
  p.win = window_of(cache, layer);
  p.c = c.decision_bias;
  p.n = n;
  p.units = L.units;
  p.hkv = c.num_kv_heads;
  p.hq = c.num_q_heads;
  p.maxpages = L.maxpages;
  p.log2p = ilog2(c.page_size);
  p.omega_src = c.omega_src;
  p.decision_src = c.decision_src;
  p.max_prompt = L.max_prompt;
  p.prompt_chunks = L.prompt_chunks;
  p.carry_blocks = L.carry_blocks;
  return DMC_OK;
}

}  // namespace

dmc_status dmc_prefill_compress(dmc_cache *cache, int32_t layer, const void *k,
                                const int64_t k_strides[3], const void *v,
                                const int64_t v_strides[3], const void *q,
                                const int64_t q_strides[3], int32_t n,
                                const int32_t *prompt_lens, int32_t *slot_index,
                                dmc_stream_t stream) {
  dmc::PrefillParams p;
  dmc_status st = prefill_params(cache, layer, k, k_strides, v, v_strides, q, q_strides, n,
                                 prompt_lens, slot_index, false, &p);
  if (st != DMC_OK) return st;
  DeviceGuard g(cache->device);
  if (!g.ok) return fail(DMC_ERR_HIP, "cannot select the cache's device");
  hipError_t e = dmc::launch_prefill(elem_bytes(cache->cfg), cache->cfg.head_dim, cache->lay.v_trans,
                                     p, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "prefill launch");
  return DMC_OK;
}

dmc_status dmc_prefill_attend(dmc_cache *cache, int32_t layer, const void *k,
                              const int64_t k_strides[3], const void *v,
                              const int64_t v_strides[3], const void *q,
                              const int64_t q_strides[3], int32_t n,
                              const int32_t *prompt_lens, void *out,
                              const int64_t out_strides[3], int32_t *slot_index,
                              dmc_stream_t stream) {
  dmc::PrefillParams p;
  dmc_status st = prefill_params(cache, layer, k, k_strides, v, v_strides, q, q_strides, n,
                                 prompt_lens, slot_index, true, &p);
  if (st != DMC_OK) return st;
  if (n > 0) {
    if (!out || !out_strides) return fail(DMC_ERR_INVALID_ARG, "out and out_strides must be non-NULL");
    if (!aligned16(out)) return fail(DMC_ERR_INVALID_ARG, "out must be 16-byte aligned");
    for (int i = 0; i < 3; ++i)
      if (out_strides[i] < 0 || out_strides[i] % 8)
        return fail(DMC_ERR_INVALID_ARG, "out strides must be non-negative multiples of 8");
  }
  const dmc_cache_config &c = cache->cfg;
  const dmc::Layout &L = cache->lay;
  if (c.dtype == DMC_BF16 && (int64_t(n) + c.page_size - 1) / c.page_size > dmc::kPromptMaxPages)
    return fail(DMC_ERR_UNSUPPORTED, "prompt of %d tokens exceeds %d pages per unit", n,
                dmc::kPromptMaxPages);
  // Windowed open states need no carry records (they span at most w tokens).
  p.carry = L.window > 0 ? nullptr : at<float>(cache, L.pf_carry);
  dmc::PromptParams a{};
  a.pool = p.pool;
  a.page_bytes = p.page_bytes;
  a.ptab = p.ptab;
  a.q = q;
  a.k = k;
  a.v = v;
  for (int i = 0; i < 3; ++i) {
    a.qs[i] = p.qs[i];
    a.ks[i] = p.ks[i];
    a.vs[i] = p.vs[i];
    a.os[i] = n > 0 ? out_strides[i] : 0;
  }
  a.out = out;
  a.prompt_lens = prompt_lens;
  a.alpha = p.alpha;
  a.omega = p.omega;
  a.count = p.count;
  a.page_base = p.page_base;
  a.carry = p.carry;
  a.scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(double(c.head_dim)));
  a.n = n;
  a.units = L.units;
  a.hkv = c.num_kv_heads;
  a.hq = c.num_q_heads;
  a.maxpages = L.maxpages;
  a.log2p = p.log2p;
  a.max_prompt = L.max_prompt;
  a.prompt_chunks = L.prompt_chunks;
  a.carry_blocks = L.carry_blocks;
  a.window = L.window;
  DeviceGuard g(cache->device);
  if (!g.ok) return fail(DMC_ERR_HIP, "cannot select the cache's device");
  const hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = dmc::launch_prefill(elem_bytes(c), c.head_dim, L.v_trans, p, s);
  if (e != hipSuccess) return hip_fail(e, "prefill launch");
  e = dmc::launch_prompt_attend(elem_bytes(c), c.head_dim, L.group, L.v_trans, a, p.ctrl, s);
  if (e != hipSuccess) return hip_fail(e, "prompt attention launch");
  return DMC_OK;
}

dmc_status dmc_cache_lengths(const dmc_cache *cache, int32_t layer, int32_t *lengths,
                             dmc_stream_t stream) {
  dmc_status st = check_layer(cache, layer);
  if (st != DMC_OK) return st;
  if (!lengths) return fail(DMC_ERR_INVALID_ARG, "lengths is NULL");
  DeviceGuard g(cache->device);
  if (!g.ok) return fail(DMC_ERR_HIP, "cannot select the cache's device");
  hipError_t e = dmc::launch_copy_i32(lengths, lens_of(cache, layer, 0),
                                      cache->lay.units, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "lengths copy");
  return DMC_OK;
}

static dmc::DenseParams dense_params(const dmc_cache *cache, int32_t layer, int32_t dense_slots) {
  const dmc::Layout &L = cache->lay;
  dmc::DenseParams p{};
  p.pool = cache->ws + L.pool;
  p.page_bytes = L.page_bytes;
  p.num_pages = cache->cfg.num_pages;
  p.ptab = at<int32_t>(cache, L.ptab) + size_t(layer) * L.units * L.maxpages;
  p.len = lens_of(cache, layer, 0);
  p.z = at<float>(cache, L.z) + size_t(layer) * L.units;
  p.ctrl = at<dmc::Control>(cache, L.ctrl);
  p.page_base = at<int32_t>(cache, L.pf_pagebase);
  p.dense_slots = dense_slots;
  p.units = L.units;
  p.maxpages = L.maxpages;
  p.log2p = ilog2(cache->cfg.page_size);
  p.max_slots = cache->cfg.max_slots_per_seq;
  return p;
}

dmc_status dmc_cache_export(const dmc_cache *cache, int32_t layer, void *k_dense, void *v_dense,
                            int32_t dense_slots, float *z, dmc_stream_t stream) {
  dmc_status st = check_layer(cache, layer);
  if (st != DMC_OK) return st;
  if (dense_slots < 0) return fail(DMC_ERR_INVALID_ARG, "dense_slots must be >= 0");
  if (!z || (dense_slots > 0 && (!k_dense || !v_dense)))
    return fail(DMC_ERR_INVALID_ARG, "k_dense, v_dense and z must be non-NULL");
  if (!aligned16(k_dense) || !aligned16(v_dense))
    return fail(DMC_ERR_INVALID_ARG, "dense tensors must be 16-byte aligned");
  dmc::DenseParams p = dense_params(cache, layer, dense_slots);
  p.kd = k_dense;
  p.vd = v_dense;
  p.z_out = z;
  DeviceGuard g(cache->device);
  if (!g.ok) return fail(DMC_ERR_HIP, "cannot select the cache's device");
  hipError_t e = dmc::launch_export(elem_bytes(cache->cfg), cache->cfg.head_dim, cache->lay.v_trans, p,
                                    static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "export launch");
  return DMC_OK;
}

dmc_status dmc_cache_import(dmc_cache *cache, int32_t layer, const void *k_dense,
                            const void *v_dense, int32_t dense_slots, const int32_t *lengths,
                            const float *z, dmc_stream_t stream) {
  dmc_status st = check_layer(cache, layer);
  if (st != DMC_OK) return st;
  if (dense_slots < 0) return fail(DMC_ERR_INVALID_ARG, "dense_slots must be >= 0");
  if (!lengths || !z || (dense_slots > 0 && (!k_dense || !v_dense)))
    return fail(DMC_ERR_INVALID_ARG, "k_dense, v_dense, lengths and z must be non-NULL");
  if (!aligned16(k_dense) || !aligned16(v_dense))
    return fail(DMC_ERR_INVALID_ARG, "dense tensors must be 16-byte aligned");
  if (cache->lay.window > 0)
    return fail(DMC_ERR_UNSUPPORTED,
                "a cache with a window keeps its open segments' raw tokens; slots cannot supply them");
  dmc::DenseParams p = dense_params(cache, layer, dense_slots);
  p.kd = const_cast<void *>(k_dense);
  p.vd = const_cast<void *>(v_dense);
  p.lengths_in = lengths;
  p.z_in = z;
  DeviceGuard g(cache->device);
  if (!g.ok) return fail(DMC_ERR_HIP, "cannot select the cache's device");
  hipError_t e = dmc::launch_import(elem_bytes(cache->cfg), cache->cfg.head_dim, cache->lay.v_trans, p,
                                    static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "import launch");
  return DMC_OK;
}

namespace {

dmc_status validate_train(const dmc_train_config *c) {
  if (!c) return fail(DMC_ERR_INVALID_ARG, "config is NULL");
  if (c->batch < 1 || c->seq_len < 1 || c->num_q_heads < 1 || c->num_kv_heads < 1)
    return fail(DMC_ERR_INVALID_ARG, "batch, seq_len and head counts must be >= 1");
  if (c->num_q_heads % c->num_kv_heads != 0)
    return fail(DMC_ERR_INVALID_ARG, "num_q_heads (%d) must be a multiple of num_kv_heads (%d)",
                c->num_q_heads, c->num_kv_heads);
  const int G = c->num_q_heads / c->num_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(DMC_ERR_UNSUPPORTED, "query group size %d not in {1,2,4,8}", G);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(DMC_ERR_UNSUPPORTED, "head_dim %d not in {64,128}", c->head_dim);
  if (c->dtype != DMC_BF16 && c->dtype != DMC_FP32)
    return fail(DMC_ERR_INVALID_ARG, "unknown dtype %d", c->dtype);
  if (!std::isfinite(c->decision_bias)) return fail(DMC_ERR_INVALID_ARG, "decision_bias not finite");
  if (!(c->temperature > 0.0f) || !std::isfinite(c->temperature))
    return fail(DMC_ERR_INVALID_ARG, "temperature must be a finite value > 0");
  if (c->window < 1 || c->window > dmc::kMaxWindow)
    return fail(DMC_ERR_INVALID_ARG, "training window %d outside [1, %d]", c->window, dmc::kMaxWindow);
  if (c->omega_src != DMC_OMEGA_LEAD_QHEAD && c->omega_src != DMC_OMEGA_UNIFORM)
    return fail(DMC_ERR_UNSUPPORTED, "training omega_src must be LEAD_QHEAD or UNIFORM");
  const int64_t rows = int64_t(c->batch) * c->seq_len * c->num_q_heads;
  if (rows > (int64_t(1) << 31) / c->head_dim)
    return fail(DMC_ERR_UNSUPPORTED, "tensors larger than 2^31 elements");
  return DMC_OK;
}

int train_elem_bytes(const dmc_train_config &c) { return c.dtype == DMC_FP32 ? 4 : 2; }

// Device that holds a training workspace (the configuration names none).
dmc_status workspace_device(const void *ws, int *dev) {
  hipPointerAttribute_t attr{};
  hipError_t e = hipPointerGetAttributes(&attr, ws);
  if (e != hipSuccess) return hip_fail(e, "hipPointerGetAttributes(workspace)");
  if (attr.type != hipMemoryTypeDevice)
    return fail(DMC_ERR_INVALID_ARG, "the training workspace is not device memory");
  *dev = attr.device;
  return DMC_OK;
}

dmc::TrainLayout train_layout_of(const dmc_train_config &c) {
  return dmc::train_layout(c.batch, c.seq_len, c.num_q_heads, c.num_kv_heads, c.head_dim,
                           train_elem_bytes(c), c.window);
}

// Common checks and parameter set-up of the two training entry points.
dmc_status train_params(const dmc_train_config *cfg, const void *q, const void *k, const void *v,
                        const float *noise, void *ws, size_t bytes, dmc::TrainParams *p) {
  dmc_status st = validate_train(cfg);
  if (st != DMC_OK) return st;
  if (!q || !k || !v || !noise || !ws)
    return fail(DMC_ERR_INVALID_ARG, "q, k, v, noise and workspace must be non-NULL");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v))
    return fail(DMC_ERR_INVALID_ARG, "q, k and v must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(ws) & 255u)
    return fail(DMC_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
  const dmc::TrainLayout L = train_layout_of(*cfg);
  if (bytes < L.total)
    return fail(DMC_ERR_INVALID_ARG, "workspace has %zu bytes, needs %zu", bytes, L.total);
  char *w = static_cast<char *>(ws);
  *p = dmc::TrainParams{};
  p->q = q;
  p->k = k;
  p->v = v;
  p->noise = noise;
  p->ks = w + L.ks;
  p->vs = w + L.vs;
  p->alpha = reinterpret_cast<float *>(w + L.alpha);
  p->omega = reinterpret_cast<float *>(w + L.omega);
  p->z = reinterpret_cast<float *>(w + L.z);
  p->mask = reinterpret_cast<float *>(w + L.mask);
  p->lse = reinterpret_cast<float *>(w + L.lse);
  p->dsum = reinterpret_cast<float *>(w + L.dsum);
  p->dks = reinterpret_cast<float *>(w + L.dks);
  p->dvs = reinterpret_cast<float *>(w + L.dvs);
  p->dmask = reinterpret_cast<float *>(w + L.dmask);
  p->qs = reinterpret_cast<float *>(w + L.qs);
  p->e = reinterpret_cast<float *>(w + L.e);
  p->c = cfg->decision_bias;
  p->tau = cfg->temperature;
  p->scale_log2 = static_cast<float>(1.4426950408889634 / std::sqrt(double(cfg->head_dim)));
  p->batch = cfg->batch;
  p->n = cfg->seq_len;
  p->hq = cfg->num_q_heads;
  p->hkv = cfg->num_kv_heads;
  p->window = cfg->window;
  p->omega_src = cfg->omega_src;
  return DMC_OK;
}

}  // namespace

size_t dmc_train_workspace_bytes(const dmc_train_config *cfg) {
  if (validate_train(cfg) != DMC_OK) return 0;
  return train_layout_of(*cfg).total;
}

dmc_status dmc_train_forward(const dmc_train_config *cfg, const void *q, const void *k,
                             const void *v, const float *noise, void *out, float *alpha,
                             void *ws, size_t bytes, dmc_stream_t stream) {
  dmc::TrainParams p;
  dmc_status st = train_params(cfg, q, k, v, noise, ws, bytes, &p);
  if (st != DMC_OK) return st;
  if (!out) return fail(DMC_ERR_INVALID_ARG, "out must be non-NULL");
  if (!aligned16(out)) return fail(DMC_ERR_INVALID_ARG, "out must be 16-byte aligned");
  p.out = out;
  p.alpha_out = alpha;
  int dev = 0;
  st = workspace_device(ws, &dev);
  if (st != DMC_OK) return st;
  DeviceGuard g(dev);   // enqueue on the workspace's device, restoring the caller's
  if (!g.ok) return fail(DMC_ERR_HIP, "cannot select the workspace's device");
  hipError_t e = dmc::launch_train_forward(train_elem_bytes(*cfg), cfg->head_dim,
                                           cfg->num_q_heads / cfg->num_kv_heads, p,
                                           static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "training forward launch");
  return DMC_OK;
}

dmc_status dmc_train_backward(const dmc_train_config *cfg, const void *q, const void *k,
                              const void *v, const float *noise, const void *out,
                              const void *dout, const float *dalpha, void *dq, void *dk, void *dv,
                              void *ws, size_t bytes, dmc_stream_t stream) {
  dmc::TrainParams p;
  dmc_status st = train_params(cfg, q, k, v, noise, ws, bytes, &p);
  if (st != DMC_OK) return st;
  if (!out || !dout || !dq || !dk || !dv)
    return fail(DMC_ERR_INVALID_ARG, "out, dout, dq, dk and dv must be non-NULL");
  if (!aligned16(out) || !aligned16(dout) || !aligned16(dq) || !aligned16(dk) || !aligned16(dv))
    return fail(DMC_ERR_INVALID_ARG, "out, dout, dq, dk and dv must be 16-byte aligned");
  p.out = const_cast<void *>(out);
  p.dout = dout;
  p.dalpha = dalpha;
  p.dq = dq;
  p.dk = dk;
  p.dv = dv;
  int dev = 0;
  st = workspace_device(ws, &dev);
  if (st != DMC_OK) return st;
  DeviceGuard g(dev);
  if (!g.ok) return fail(DMC_ERR_HIP, "cannot select the workspace's device");
  hipError_t e = dmc::launch_train_backward(train_elem_bytes(*cfg), cfg->head_dim,
                                            cfg->num_q_heads / cfg->num_kv_heads, p,
                                            static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "training backward launch");
  return DMC_OK;
}

static dmc_status read_control(dmc_cache *cache, dmc_stream_t stream, dmc::Control *out) {
  DeviceGuard g(cache->device);
  if (!g.ok) return fail(DMC_ERR_HIP, "cannot select the cache's device");
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  e = hipMemcpy(out, cache->ws + cache->lay.ctrl, sizeof(dmc::Control), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "reading the control block");
  return DMC_OK;
}

dmc_status dmc_cache_check(dmc_cache *cache, dmc_stream_t stream) {
  if (!cache) return fail(DMC_ERR_INVALID_ARG, "cache is NULL");
  dmc::Control ctl{};
  dmc_status st = read_control(cache, stream, &ctl);
  if (st != DMC_OK) return st;
  if (ctl.flags & (dmc::FLAG_POOL_EXHAUSTED | dmc::FLAG_SLOTS_EXHAUSTED))
    return fail(DMC_ERR_CAPACITY, "cache capacity exhausted (flags 0x%x: %s%s)", ctl.flags,
                (ctl.flags & dmc::FLAG_POOL_EXHAUSTED) ? "page pool " : "",
                (ctl.flags & dmc::FLAG_SLOTS_EXHAUSTED) ? "slots per unit" : "");
  if (ctl.flags & dmc::FLAG_BAD_LENGTH)
    return fail(DMC_ERR_INVALID_ARG, "an imported or prompt length was out of range");
  return DMC_OK;
}

dmc_status dmc_cache_pages_used(dmc_cache *cache, int64_t *pages_out, dmc_stream_t stream) {
  if (!cache || !pages_out) return fail(DMC_ERR_INVALID_ARG, "cache and pages_out must be non-NULL");
  dmc::Control ctl{};
  dmc_status st = read_control(cache, stream, &ctl);
  if (st != DMC_OK) return st;
  const unsigned long long used = ctl.pages_used;
  const unsigned long long cap = static_cast<unsigned long long>(cache->cfg.num_pages);
  *pages_out = static_cast<int64_t>(used < cap ? used : cap);
  return DMC_OK;
}

}  // extern "C"
