// Internal declarations shared by the host API (dmc_api.cpp) and the gfx950
// kernels (dmc_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dmc {

__host__ __device__ constexpr inline size_t align_up(size_t x, size_t a) {
  return (x + a - 1) / a * a;
}

// Device flag bits (sticky until reset).
enum : int32_t {
  FLAG_POOL_EXHAUSTED = 1,   // no free page for an append
  FLAG_SLOTS_EXHAUSTED = 2,  // unit already holds max_slots_per_seq slots
  FLAG_BAD_LENGTH = 4,       // imported length or prompt length out of range
};

// Control block at the start of the control section.
struct Control {
  unsigned long long pages_used;  // bump allocator of the page pool
  long long alloc_base;           // first page of the last prefill / import allocation
  long long alloc_count;          // pages in it (0 after a failed allocation)
  int32_t flags;
  int32_t pad[9];
};

// Byte offsets of the workspace sections (all 256-byte aligned).
struct Layout {
  size_t pool, ptab, lens, z, ctrl, meta, partials, pf_alpha, pf_omega, pf_count, pf_mask,
      pf_pagebase, pf_carry, win, win_omega, win_len;
  size_t total;
  int64_t page_bytes;     // 2 * P * d * elem_bytes (K rows, then V rows)
  int32_t units;          // B * Hkv per layer
  int32_t maxpages;       // page-table width per unit
  int32_t group;          // G
  int32_t split_tile;     // cap on positions per decode range (0 = none)
  int64_t max_records;    // decode partial records: ranges + units
  int32_t max_prompt;     // prefill staging capacity (tokens)
  int32_t prompt_chunks;  // ceil(max_prompt / 64)
  int32_t carry_blocks;   // ceil(max_prompt / 32)
  int32_t window;         // window-grouping width (0 = exact Algorithm 1)
  int32_t slot_group;     // units per entry of the decode's slot-space table in LDS
  bool v_trans;           // value pages stored transposed (matrix-core decode)
};

// Window grouping: per unit, a ring of `window` raw tokens of its open
// segment (token j of the segment in entry j mod window): a key row with
// element 0 zeroed, then a value row, in the cache dtype; their omegas
// (fp32) and the open segment's token count.
struct WindowState {
  char *ring;              // [U][window][2][d] of this layer
  float *omega;            // [U][window]
  int32_t *seg_len;        // [U]
  int32_t window;          // 0 = no window
};

// Everything the decode kernel needs for one layer.
struct DecodeParams {
  char *pool;
  int64_t page_bytes;
  int64_t num_pages;
  int32_t *ptab;           // [U, maxpages] of this layer
  int32_t *len_in;         // [U] lengths before this step (the layer's current lengths)
  int32_t *len_out;        // [U] lengths after this step; the combine launch copies them
                           // back into len_in
  float *z;                // [U]
  Control *ctrl;
  const void *q, *k, *v;
  void *out;
  int32_t *slot_index;     // optional [U]
  float *partials;         // [tiles, G, d + 4]
  int32_t *meta;           // [U, 2]: first partial record, record count (for the combine)
  WindowState win;
  float c;                 // decision bias
  float scale_log2;        // log2(e) / sqrt(d)
  int32_t units, hkv, hq, maxpages, max_slots, log2p, split_tile, omega_src, decision_src;
  int32_t slot_group;      // units per entry of the slot-space table in LDS (1, or 2..64)
};

struct PrefillParams {
  char *pool;
  int64_t page_bytes;
  int64_t num_pages;
  int32_t *ptab;
  int32_t *len;            // [U] current lengths of this layer
  float *z;
  Control *ctrl;
  const void *k, *v, *q;
  int64_t ks[3], vs[3], qs[3];
  const int32_t *prompt_lens;
  int32_t *slot_index;     // optional [U, n]
  uint8_t *alpha;          // [U, max_prompt] (staged only for prompt attention / window)
  float *omega;            // [U, max_prompt] (likewise)
  int32_t *count;          // [U, prompt_chunks] segment starts per 64-token chunk
  uint64_t *mask;          // [U, prompt_chunks] bit i: token 64 c + i starts a segment
  int32_t *page_base;      // [U]
  float *carry;            // optional [U, carry_blocks, carry_stride]: open-segment sums at
                           // every 32-token boundary inside a segment (prompt attention)
  WindowState win;
  float c;
  int32_t n, units, hkv, hq, maxpages, log2p, omega_src, max_prompt, prompt_chunks,
      carry_blocks, decision_src;
};

// Floats per carry record: sum of omega * k (d), sum of omega * v (d), sum of
// omega, padding to 16 bytes.
__host__ __device__ constexpr inline int carry_stride(int head_dim) { return 2 * head_dim + 4; }

// Prompt-phase attention over a freshly compacted layer (after the prefill
// passes have run with carry records enabled).
struct PromptParams {
  const char *pool;
  int64_t page_bytes;
  const int32_t *ptab;     // [U, maxpages] of this layer
  const void *q, *k, *v;
  int64_t qs[3], ks[3], vs[3];   // element strides of (batch, token, head); d contiguous
  void *out;
  int64_t os[3];
  const int32_t *prompt_lens;
  const uint8_t *alpha;    // [U, max_prompt] decisions (1 = accumulate; 1 past the prompt)
  const float *omega;      // [U, max_prompt]
  const int32_t *count;    // [U, prompt_chunks] segment starts per 64-token chunk
  const int32_t *page_base;  // [U]; < 0 when the layer's allocation failed
  const float *carry;      // [U, carry_blocks, carry_stride(d)]
  float scale_log2;        // log2(e) / sqrt(d)
  int32_t n, units, hkv, hq, maxpages, log2p, max_prompt, prompt_chunks, carry_blocks;
  int32_t window;          // window grouping: open states over the last `window` tokens
};

struct DenseParams {
  char *pool;
  int64_t page_bytes;
  int64_t num_pages;
  int32_t *ptab;
  int32_t *len;
  float *z;
  Control *ctrl;
  void *kd, *vd;           // dense [U, dense_slots, d]
  const int32_t *lengths_in;
  const float *z_in;
  float *z_out;
  int32_t *page_base;
  int32_t dense_slots, units, maxpages, log2p, max_slots;
};

// Training-time forward/backward (Sec. 3.2 + 3.3).  Units u = b * hkv + g;
// per-unit arrays are [U][n] (or [U][n][d] for rows).
struct TrainParams {
  const void *q, *k, *v;     // [B, n, H, d] contiguous
  const float *noise;        // [B, n, Hkv]
  void *out;                 // [B, n, Hq, d]
  float *alpha_out;          // optional [B, n, Hkv]
  const void *dout;          // [B, n, Hq, d]
  const float *dalpha;       // optional [B, n, Hkv]
  void *dq, *dk, *dv;
  // workspace
  void *ks, *vs;             // unrolled states [U][n][d] (+ 32 zero rows), config dtype;
                             // key element 0 holds the state's mask entry * sqrt(d)
  float *alpha, *omega;      // per token [U][n]
  float *z;                  // state normalisers [U][n]
  float *mask;               // [U][n]: log(1 - alpha_{j+1}) for state j < n - 1
  float *lse;                // [U][n][G]: log2-sum-exp of each query row (log2 domain)
  float *dsum;               // [U][n][G]: sum(dout * out) of each query row
  float *dks, *dvs;          // gradients of the states: [U][n][d] fp32 (vector passes) or,
                             // in the same bytes, bf16 head and tail planes [2][U][n][d]
                             // (matrix-core passes)
  float *dmask;              // [U][n]
  float *qs;                 // [2][U][n]: V~_j . dV~_j, then K~_j . dK~_j (matrix-core passes)
  float *e;                  // [U][n][w]: d loss / d weight of token t in state t + i
  float c, tau, scale_log2;
  int32_t batch, n, hq, hkv, window, omega_src;
};

// Workspace layout of a training configuration.
struct TrainLayout {
  size_t ks, vs, alpha, omega, z, mask, lse, dsum, dks, dvs, dmask, qs, e, total;
};
TrainLayout train_layout(int batch, int n, int hq, int hkv, int head_dim, int elem_bytes, int window);

hipError_t launch_train_forward(int elem_bytes, int head_dim, int group, const TrainParams &p,
                                hipStream_t s);
hipError_t launch_train_backward(int elem_bytes, int head_dim, int group, const TrainParams &p,
                                 hipStream_t s);

// Launchers (return hipGetLastError() after enqueueing).
hipError_t launch_fill_i32(int32_t *p, int32_t value, size_t count, hipStream_t s);
hipError_t launch_fill_u8(void *p, size_t bytes, hipStream_t s);
hipError_t launch_copy_i32(int32_t *dst, const int32_t *src, size_t count, hipStream_t s);
// vt: value pages stored transposed ([d][32] per page; bf16, G >= 4, P == 32),
// decoded on matrix cores.
hipError_t launch_decode(int elem_bytes, int head_dim, int group, bool vt, const DecodeParams &p,
                         int grid, hipStream_t s);
hipError_t launch_prefill(int elem_bytes, int head_dim, bool vt, const PrefillParams &p,
                          hipStream_t s);
hipError_t launch_import(int elem_bytes, int head_dim, bool vt, const DenseParams &p, hipStream_t s);
hipError_t launch_export(int elem_bytes, int head_dim, bool vt, const DenseParams &p, hipStream_t s);

// Allocation-free decode (dmc_decode_step_static): the split-K records live in
// a file-scope static device array of this many bytes (dmc_kernels.hip).
// static_scratch() returns its address on the current device, resolved with
// hipGetSymbolAddress on the first call per device and kept per device.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
hipError_t static_scratch(void **ptr);

// Largest window-grouping width.
constexpr int kMaxWindow = 64;

// Largest prompt, in pages per unit, of the matrix-core prompt attention
// (its page-table slice is held in LDS).
constexpr int kPromptMaxPages = 1024;

// Prompt-phase attention; bf16 runs on matrix cores (value pages read as rows,
// or as the transposed pages of grouped-query caches), fp32 on the vector ALUs.
hipError_t launch_prompt_attend(int elem_bytes, int head_dim, int group, bool vt,
                                const PromptParams &p, const Control *ctrl, hipStream_t s);

// Dynamic LDS bytes of the decode kernel for a slot-space table of
// `table_entries` ints (ceil(units / slot_group) + 1) / group / head dim (and
// whether the cache has a window).
size_t decode_lds_bytes(int table_entries, int group, int head_dim, bool window);
// Largest units per slot-space table entry.
constexpr int kMaxSlotGroup = 64;
// Largest number of virtual slot-space positions a decode kernel appends to a
// unit (bounds the split-K ranges: S <= units * (max_slots_per_seq + this)).
constexpr int kDecodeUnitOverhead = 32;
// Static LDS of the decode kernel that runs such a cache (matrix-core kernel:
// its chunk ring and staging rows).
size_t decode_static_lds_bytes(int head_dim, bool v_trans);

}  // namespace dmc
