// gfx950 kernels of the DMC decode path.
//
// Method: Nawrot et al., "Dynamic Memory Compression" (ICML 2024).
//   Sec. 3.1 + Algorithm 1: per-head decision alpha = round(sigmoid(k[0] - c))
//   (= k[0] > c), importance omega = sigmoid(q[0]); accumulate into the last
//   slot as an omega-weighted running mean, or append a slot.
//   Sec. 3.1 (last paragraph) + Sec. 2.1: softmax attention over the ragged,
//   per-head compressed cache.  Sec. 3.3: paged storage, pages per head.
//
// Memory layout (one workspace, see dmc_api.cpp):
//   page pool: page = P key rows then P value rows, each row d contiguous
//              elements; a row is 128..512 bytes, a page 2*P*row bytes.
//   page table [L][U][maxpages] int32, lengths [2][L][U] int32 (buffer 0
//   holds the current counts; a decode step reads buffer 0 and writes its
//   post-step counts to buffer 1, so every workgroup sees the same pre-step
//   lengths, and its combine launch copies them back), z [L][U] fp32.
//
// Decode = one fused launch per layer (Algorithm 1 update + split-K
// attention, balanced by actual compressed length) plus a small combine
// launch for units split over several pieces.
#include "dmc_device.h"
#include "dmc_mfma.h"

#include <algorithm>
#include <mutex>
#include <type_traits>

namespace dmc {

// Scratch of the allocation-free decode entry point: split-K partial records
// and the per-unit record table of one decode launch.  In host code the name
// `scratch` is only a stand-in for the symbol, never a device address: the
// address on a device comes from hipGetSymbolAddress (static_scratch).  Every
// call on a GPU shares that GPU's copy; a call writes every entry it reads.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_addr[kMaxDevices] = {};
}  // namespace

hipError_t static_scratch(void **ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_addr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_addr[dev] = p;
  }
  *ptr = g_scratch_addr[dev];
  return hipSuccess;
}

namespace {

#ifndef DMC_VALU_CHUNK
#define DMC_VALU_CHUNK 16
#endif
#ifndef DMC_VALU_BUFFERS
#define DMC_VALU_BUFFERS 3
#endif
constexpr int kRangesPerWave = 1;   // slot-space ranges per decode wave (2 and 3 measured slower)
// Virtual positions appended to every unit in the slot space, standing for a
// piece's fixed cost (its page-table and first-chunk round trips, the owner's
// update), so that equal ranges carry equal cost rather than equal slots:
// 32 for the vector-ALU decode (7B stack 180.5 -> 178.9 us per call; 16 and
// 64 in between), none for the matrix-core decode, whose ranges span about
// two units of 2000+ slots (no change measured).  At most kDecodeUnitOverhead.
constexpr int kValuUnitOverhead = 32;
constexpr int kMfmaUnitOverhead = 0;
// Largest excess, in percent of the equal slot share, at which the matrix-core
// decode gives every wave whole units instead of equal slot ranges.
constexpr int kWholeUnitSlack = 10;
static_assert(kValuUnitOverhead <= kDecodeUnitOverhead && kMfmaUnitOverhead <= kDecodeUnitOverhead,
              "slot-space overhead bound");
#ifndef DMC_VALU_DECODE_WAVES
#define DMC_VALU_DECODE_WAVES 8
#endif
// Workgroup size of the vector-ALU decode.  The launch keeps the waves of the
// persistent grid (kDecodeWgPerCu workgroups of 4 waves per compute unit)
// and packs them into workgroups of this many threads; fp32 caches and groups
// of more than two query heads keep 4 waves (their registers need more than
// the 256 VGPRs per wave an 8-wave workgroup leaves).
template <int ES, int G>
constexpr int valu_decode_threads() { return ES == 2 && G <= 2 ? 64 * DMC_VALU_DECODE_WAVES : kThreads; }
static_assert(64 * DMC_VALU_DECODE_WAVES % kThreads == 0 && DMC_VALU_DECODE_WAVES <= 16, "decode workgroup");
constexpr int kValuChunk = DMC_VALU_CHUNK;  // rows per chunk of the vector-ALU decode
constexpr int kBuf = DMC_VALU_BUFFERS;      // chunk buffers in flight per wave



// ---------------------------------------------------------------------------
// Fused decode: Algorithm 1 update + split-K attention + combine.
//
// Load balance by actual compressed length: the layer's units are laid end
// to end in one "slot space" of S = sum_u max(l_u, 1) positions, cut into
// equal ranges, one per wave (at most split_tile positions each, when set).
// A range may cover the end of one unit and the start of the next; each
// (range, unit) piece keeps an online-softmax state (max, sum, acc[d]) per
// query head of the group.  The piece holding a unit's last position owns
// the open slot and runs the unit's Algorithm 1 update before attending to
// it; every other piece reads closed slots only, so the fusion is race free.
// A unit covered by one piece writes its output directly; otherwise each
// piece writes a partial record (index range + unit), combined by a second,
// small launch.  No barrier and no atomic is taken after the slot space is
// built (the page allocator's bump counter aside).
// ---------------------------------------------------------------------------


// Window grouping (Sec. 3.3): with the new token at position j of its
// segment, the open slot is the omega-weighted mean of the segment's
// positions j - m + 1 .. j, m = min(j + 1, w) -- the ring holds the earlier
// ones (entry i mod w).  Vector-ALU layout: rows of LPR lanes, each lane a
// 16-byte slice; the RPI row groups of the wave take every RPI-th ring entry
// and their sums are added across groups.  On entry ck, cv hold the new
// token's slice (key element 0 zeroed) and om its omega; on return they
// hold the mean, and the omega sum of the window is returned.
template <int ES, int LPR>
__device__ __forceinline__ float window_mean_rows(const WindowState &w, int u, int j, int grp,
                                                  int part, float *ck, float *cv, float om) {
  using V = V16<ES>;
  constexpr int VN = V::N, RB = LPR * 16, RPI = 64 / LPR, kBatch = 4;
  const int W = w.window;
  const int m = min(j + 1, W);
  const char *ring = w.ring + int64_t(u) * W * 2 * RB + part * 16;
  const float *wo = w.omega + int64_t(u) * W;
  float sk[VN], sv[VN], zs = 0.0f;
#pragma unroll
  for (int e = 0; e < VN; ++e) sk[e] = sv[e] = 0.0f;
  for (int i0 = j - m + 1 + grp; i0 < j; i0 += kBatch * RPI) {
    uint4 kr[kBatch], vr[kBatch];
    float wt[kBatch];
#pragma unroll
    for (int q = 0; q < kBatch; ++q) {
      const int i = i0 + q * RPI;
      const int ent = (i < j ? i : j - 1) % W;   // past the window: any entry, weight 0
      kr[q] = ld16(ring + int64_t(ent) * 2 * RB);
      vr[q] = ld16(ring + int64_t(ent) * 2 * RB + RB);
      wt[q] = i < j ? wo[ent] : 0.0f;
    }
#pragma unroll
    for (int q = 0; q < kBatch; ++q) {
      float kf[VN], vf[VN];
      V::unpack(kr[q], kf);
      V::unpack(vr[q], vf);
#pragma unroll
      for (int e = 0; e < VN; ++e) {
        sk[e] = fmaf(wt[q], kf[e], sk[e]);
        sv[e] = fmaf(wt[q], vf[e], sv[e]);
      }
      zs += wt[q];
    }
  }
#pragma unroll
  for (int o = LPR; o < 64; o <<= 1) {
#pragma unroll
    for (int e = 0; e < VN; ++e) {
      sk[e] += __shfl_xor(sk[e], o, 64);
      sv[e] += __shfl_xor(sv[e], o, 64);
    }
    zs += __shfl_xor(zs, o, 64);
  }
  zs += om;
  const float inv = 1.0f / zs;
#pragma unroll
  for (int e = 0; e < VN; ++e) {
    ck[e] = fmaf(om, ck[e], sk[e]) * inv;
    cv[e] = fmaf(om, cv[e], sv[e]) * inv;
  }
  return zs;
}

// Merge (m2, l2, a2) into (m, l, a); scores are in the log2 domain.
template <int N>
__device__ __forceinline__ void merge_state(float &m, float &l, float *a, float m2, float l2,
                                            const float *a2) {
  const float mn = fmaxf(m, m2);
  if (mn == neg_inf()) return;
  const float s1 = fast_exp2(m - mn), s2 = fast_exp2(m2 - mn);
  l = l * s1 + l2 * s2;
#pragma unroll
  for (int e = 0; e < N; ++e) a[e] = a[e] * s1 + a2[e] * s2;
  m = mn;
}


// Slot space of a layer: unit u owns positions [off_u, off_u + n_u) with
// n_u = max(l_u, 1) + OVH (pre-step lengths, OVH virtual positions for the
// piece's fixed cost); position off_u + max(l_u, 1) - 1 is the unit's open
// slot (or, for an empty unit, the slot its first token opens), and the piece
// holding the unit's last position owns it.
// Every workgroup builds the exclusive prefix in LDS and gets S.  The table
// holds every unit's offset (s_off[0..U]); layers whose full table would not
// fit in LDS run the GRP kernels, which keep only every g-th entry (g =
// p.slot_group, a power of two <= 64): s_off[j] = off of unit j g, for
// j <= NG = ceil(U / g), s_off[NG] = S.
template <bool GRP, int OVH, int NT = kThreads>
__device__ __forceinline__ int build_slot_space(const DecodeParams &p, int *s_off, int *s_wsum) {
  constexpr int NW = NT / 64;
  const int U = p.units, g = GRP ? p.slot_group : 1, NG = (U + g - 1) / g;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int kBatch = 8;     // coalesced loads in flight per thread
  for (int i0 = 0; i0 < U; i0 += NT * kBatch) {
    int v[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = i0 + j * NT + tid;
      v[j] = i < U ? p.len_in[i] : 0;
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = i0 + j * NT + tid;   // units of a wave are 64 consecutive ones
      int n = i < U ? max(v[j], 1) + OVH : 0;
      for (int o = 1; o < g; o <<= 1) n += __shfl_xor(n, o, 64);   // sum over the g-unit group
      if (i < U && (i & (g - 1)) == 0) s_off[i / g] = n;
    }
  }
  __syncthreads();
  const int per = (NG + NT - 1) / NT;
  const int i0 = min(tid * per, NG), i1 = min(i0 + per, NG);
  int sum = 0;
  for (int i = i0; i < i1; ++i) sum += s_off[i];
  int incl = sum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(incl, o, 64);
    if (lane >= o) incl += t;
  }
  if (lane == 63) s_wsum[wave] = incl;
  __syncthreads();
  int run = incl - sum, total = 0;
  for (int w = 0; w < NW; ++w) {
    if (w < wave) run += s_wsum[w];
    total += s_wsum[w];
  }
  for (int i = i0; i < i1; ++i) {
    const int n = s_off[i];
    s_off[i] = run;
    run += n;
  }
  if (tid == 0) s_off[NG] = total;
  __syncthreads();
  return s_off[NG];
}

// Unit holding slot-space position pos (off_u <= pos < off_u + n_u); its
// offset goes to `off`.  Grouped tables: the group by binary search, then the
// unit inside it from the group's lengths (one wave-wide load, a scan).
template <bool GRP, int OVH>
__device__ __forceinline__ int unit_at(const DecodeParams &p, const int *s_off, int pos, int &off) {
  const int U = p.units, g = GRP ? p.slot_group : 1, NG = (U + g - 1) / g;
  int lo = 0, hi = NG - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (s_off[mid] <= pos) lo = mid; else hi = mid - 1;
  }
  off = s_off[lo];
  if (!GRP) return lo;
  const int lane = threadIdx.x & 63, u0 = lo * g;
  const int n = (lane < g && u0 + lane < U) ? max(p.len_in[u0 + lane], 1) + OVH : 0;
  int incl = n;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(incl, o, 64);
    if (lane >= o) incl += t;
  }
  const int jl = __ffsll(static_cast<long long>(__ballot(lane < g && off + incl > pos))) - 1;
  off += __shfl(incl - n, jl, 64);
  return u0 + jl;
}

template <int ES, int D, int G, bool WIN, bool GRP>
__global__ __launch_bounds__((valu_decode_threads<ES, G>())) void decode_kernel(DecodeParams p) {
  constexpr int NT = valu_decode_threads<ES, G>(), NW = NT / 64;   // threads, waves per workgroup
  using V = V16<ES>;
  constexpr int VN = V::N;        // elements per 16-byte lane chunk
  constexpr int LPR = D / VN;     // lanes per cache row
  constexpr int RPI = 64 / LPR;   // rows per wave-wide load
  constexpr int NI = kValuChunk / RPI;
  constexpr int REC = D + 4;      // partial record: m, l, -, -, acc[D]
  constexpr int RB = D * ES;      // bytes per row
  constexpr int kLog2Chunk = kValuChunk == 8 ? 3 : kValuChunk == 16 ? 4 : 5;
  static_assert(kValuChunk == (1 << kLog2Chunk) && NI >= 1, "chunk rows");

  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int s_wsum[NW];
  int *s_off = reinterpret_cast<int *>(smem);   // slot-space table (build_slot_space)

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int grp = lane / LPR, part = lane % LPR;
  const int P = 1 << p.log2p;
  const int CS = P < kValuChunk ? P : kValuChunk;
  const int log2cs = p.log2p < kLog2Chunk ? p.log2p : kLog2Chunk;

  constexpr int OVH = kValuUnitOverhead;
  const int S = build_slot_space<GRP, OVH, NT>(p, s_off, s_wsum);
  const int nwaves = gridDim.x * NW;
  int span = (S + kRangesPerWave * nwaves - 1) / (kRangesPerWave * nwaves);   // equal shares
  if (p.split_tile > 0 && span > p.split_tile) span = p.split_tile;
  const int nranges = (S + span - 1) / span;

  for (int r = blockIdx.x * NW + wave; r < nranges; r += nwaves) {
    int pos = r * span;
    const int pos_end = min(pos + span, S);
    int off;   // the piece's unit's offset; a later piece of the range starts its unit
    for (int u = unit_at<GRP, OVH>(p, s_off, pos, off); pos < pos_end; ++u, off = pos) {
      if constexpr (!GRP) off = s_off[u];
      const int n_u = GRP ? max(p.len_in[u], 1) + OVH : s_off[u + 1] - off;
      const int start = pos - off;
      const int stop = min(pos_end, off + n_u) - off;   // this piece: [start, stop)
      pos = off + stop;
      const bool owner = stop == n_u;                   // holds the open slot
      const int l = p.len_in[u];
      const int b = u / p.hkv, g = u - b * p.hkv;
      const int64_t pt = int64_t(u) * p.maxpages;
      // closed slots [start, end): the open slot and the virtual tail are not streamed
      int end = min(owner ? n_u - 1 : stop, n_u - OVH - 1);

      // The unit's query heads (this lane's slice), element 0 zeroed.  Scores
      // are scaled by log2(e)/sqrt(d) after the row sum.
      QSlice<ES> qs[G];
#pragma unroll
      for (int h = 0; h < G; ++h)
        qs[h].load(static_cast<const char *>(p.q) +
                       (int64_t(b * p.hq + g * G + h) * D + part * VN) * ES,
                   part == 0);

      // Owner of the unit's last position: start the loads Algorithm 1 needs
      // (new key/value, decision and importance neurons, z, the open slot) so
      // they are in flight while the closed slots stream; the update itself
      // runs after the loop.  The loop covers [start, n_u - 1) only; the open
      // slot is attended to after the update, as merged or as it was.
      uint4 k_raw = make_uint4(0, 0, 0, 0), v_raw = k_raw, ok_raw = k_raw, ov_raw = k_raw;
      float k0 = 0.0f, q0 = 0.0f, zold = 0.0f;
      int open_page = -1, seg_len = 0;
      if (owner) {
        const int dg = p.decision_src ? 0 : g;   // head whose neurons decide for this unit
        if (WIN && l > 0) seg_len = p.win.seg_len[u];
        k0 = load_elem<ES>(p.k, int64_t(b * p.hkv + dg) * D);
        q0 = load_elem<ES>(p.q, int64_t(b * p.hq + dg * G) * D);
        k_raw = ld16(static_cast<const char *>(p.k) + (int64_t(u) * D + part * VN) * ES);
        v_raw = ld16(static_cast<const char *>(p.v) + (int64_t(u) * D + part * VN) * ES);
        if (l > 0) {
          zold = p.z[u];
          open_page = p.ptab[pt + ((l - 1) >> p.log2p)];
          const char *kr = p.pool + int64_t(open_page) * p.page_bytes +
                           int64_t((l - 1) & (P - 1)) * RB + part * 16;
          ok_raw = ld16(kr);
          ov_raw = ld16(kr + int64_t(P) * RB);
        }
      }

      // Attention over the closed slots [start, end) of this piece.
      float m[G], ls[G], acc[G][VN];
#pragma unroll
      for (int h = 0; h < G; ++h) {
        m[h] = neg_inf();
        ls[h] = 0.0f;
#pragma unroll
        for (int e = 0; e < VN; ++e) acc[h][e] = 0.0f;
      }
      if (end > start) {
        // Chunks of <= CS rows inside one page, kBuf register buffers in a
        // ring: kBuf - 1 chunks are in flight while one is consumed.
        const int c0 = start >> log2cs, c1 = (end - 1) >> log2cs;
        auto issue = [&](int ch, uint4 *kr, uint4 *vr) {
          const int row0 = ch << log2cs;
          const int rlo = max(start, row0) - row0, rhi = min(end, row0 + CS) - row0;
          const int page = p.ptab[pt + (row0 >> p.log2p)];
          const char *kb = p.pool + int64_t(page) * p.page_bytes + int64_t(row0 & (P - 1)) * RB +
                           part * 16;
          const char *vb = kb + int64_t(P) * RB;
#pragma unroll
          for (int i = 0; i < NI; ++i) {
            const int rr = min(max(i * RPI + grp, rlo), rhi - 1);
            kr[i] = ld16_stream(kb + rr * RB);
          }
#pragma unroll
          for (int i = 0; i < NI; ++i) {
            const int rr = min(max(i * RPI + grp, rlo), rhi - 1);
            vr[i] = ld16_stream(vb + rr * RB);
          }
        };
        auto consume = [&](int ch, const uint4 *kr, const uint4 *vr) {
          const int row0 = ch << log2cs;
          const int rlo = max(start, row0) - row0, rhi = min(end, row0 + CS) - row0;
          float s[G][NI];
#pragma unroll
          for (int i = 0; i < NI; ++i) {
            const int rr = i * RPI + grp;
            const bool valid = rr >= rlo && rr < rhi;
#pragma unroll
            for (int h = 0; h < G; ++h) {
              const float d = row_sum<LPR>(qs[h].dot(kr[i])) * p.scale_log2;
              s[h][i] = valid ? d : neg_inf();
            }
          }
          float mn[G];
#pragma unroll
          for (int h = 0; h < G; ++h) {
            float mc = s[h][0];
#pragma unroll
            for (int i = 1; i < NI; ++i) mc = fmaxf(mc, s[h][i]);
            mn[h] = fmaxf(m[h], mc);
            if (mn[h] != neg_inf()) {
              const float sc = fast_exp2(m[h] - mn[h]);
              ls[h] *= sc;
#pragma unroll
              for (int e = 0; e < VN; ++e) acc[h][e] *= sc;
#pragma unroll
              for (int i = 0; i < NI; ++i) {
                s[h][i] = fast_exp2(s[h][i] - mn[h]);
                ls[h] += s[h][i];
              }
              m[h] = mn[h];
            }
          }
#pragma unroll
          for (int i = 0; i < NI; ++i) {
            float vf[VN];
            V::unpack(vr[i], vf);
#pragma unroll
            for (int h = 0; h < G; ++h) {
              if (mn[h] == neg_inf()) continue;
#pragma unroll
              for (int e = 0; e < VN; ++e) acc[h][e] = fmaf(s[h][i], vf[e], acc[h][e]);
            }
          }
        };
        uint4 kbuf[kBuf][NI], vbuf[kBuf][NI];
#pragma unroll
        for (int j = 0; j < kBuf - 1; ++j)
          if (c0 + j <= c1) issue(c0 + j, kbuf[j], vbuf[j]);
        for (int ch = c0; ch <= c1; ch += kBuf) {
#pragma unroll
          for (int j = 0; j < kBuf; ++j) {
            if (ch + j > c1) break;
            if (ch + j + kBuf - 1 <= c1)
              issue(ch + j + kBuf - 1, kbuf[(j + kBuf - 1) % kBuf], vbuf[(j + kBuf - 1) % kBuf]);
            consume(ch + j, kbuf[j], vbuf[j]);
          }
        }
      }

      // Merge the RPI row groups of the wave.
#pragma unroll
      for (int o = LPR; o < 64; o <<= 1) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
          float a2[VN];
#pragma unroll
          for (int e = 0; e < VN; ++e) a2[e] = __shfl_xor(acc[h][e], o, 64);
          const float m2 = __shfl_xor(m[h], o, 64), l2 = __shfl_xor(ls[h], o, 64);
          merge_state<VN>(m[h], ls[h], acc[h], m2, l2, a2);
        }
      }

      if (owner) {
        // Algorithm 1 for unit u: alpha from k[0] (the first token of an empty
        // unit appends), omega from q[0]; k[0] <- 0; merge or append.
        const int alpha = (l > 0 && k0 > p.c) ? 1 : 0;
        float om;
        if (p.omega_src == 0) {
          om = sigmoid_floor(q0);
        } else if (p.omega_src == 1) {
          const int dg = p.decision_src ? 0 : g;
          float sum = 0.0f;
          for (int h = 0; h < G; ++h)
            sum += sigmoid_floor(load_elem<ES>(p.q, int64_t(b * p.hq + dg * G + h) * D));
          om = fmaxf(sum / G, 0x1p-100f);
        } else {
          om = 1.0f;   // uniform weighting
        }
        float ck[VN], cv[VN];
        V::unpack(k_raw, ck);
        V::unpack(v_raw, cv);
        if (part == 0) ck[0] = 0.0f;
        int flag = 0, slot, page = open_page;
        bool has_cur = true;
        float znew;
        if (WIN && alpha) {   // window grouping: mean of the last w tokens
          slot = l - 1;
          znew = window_mean_rows<ES, LPR>(p.win, u, seg_len, grp, part, ck, cv, om);
        } else if (alpha) {
          float ok[VN], ov[VN];
          V::unpack(ok_raw, ok);
          V::unpack(ov_raw, ov);
          slot = l - 1;
          znew = zold + om;
#pragma unroll
          for (int e = 0; e < VN; ++e) {
            ck[e] = (ok[e] * zold + ck[e] * om) / znew;
            cv[e] = (ov[e] * zold + cv[e] * om) / znew;
          }
        } else {
          if (l > 0) {   // the old open slot stays as it is: attend to it
            float ov[VN];
            V::unpack(ov_raw, ov);
#pragma unroll
            for (int h = 0; h < G; ++h) {
              const float d = row_sum<LPR>(qs[h].dot(ok_raw)) * p.scale_log2;
              merge_state<VN>(m[h], ls[h], acc[h], d, 1.0f, ov);
            }
          }
          slot = l;
          znew = om;
          if (l >= p.max_slots) {
            has_cur = false;
            flag = FLAG_SLOTS_EXHAUSTED;
          } else if ((l & (P - 1)) == 0) {
            int pg = 0;
            if (lane == 0) {
              const unsigned long long x = atomicAdd(&p.ctrl->pages_used, 1ull);
              pg = x < static_cast<unsigned long long>(p.num_pages) ? static_cast<int>(x) : -1;
            }
            pg = __shfl(pg, 0, 64);
            if (pg < 0) {
              has_cur = false;
              flag = FLAG_POOL_EXHAUSTED;
            } else {
              page = pg;
              if (lane == 0) p.ptab[pt + (l >> p.log2p)] = pg;
            }
          }
          // otherwise slot l shares the open slot's page
        }
        if (WIN && has_cur) {   // the token joins its segment's window ring
          const int W = p.win.window, j = alpha ? seg_len : 0, ent = j % W;
          if (grp == 0) {
            uint4 kh = k_raw;
            if (part == 0) kh.x &= ES == 2 ? 0xffff0000u : 0u;   // k_t[0] <- 0
            char *er = p.win.ring + (int64_t(u) * W + ent) * 2 * RB + part * 16;
            st16(er, kh);
            st16(er + RB, v_raw);
          }
          if (lane == 0) {
            p.win.omega[int64_t(u) * W + ent] = om;
            p.win.seg_len[u] = j + 1;
          }
        }
        if (has_cur) {
          const uint4 kp = V::pack(ck), vp = V::pack(cv);   // ck, cv become the stored values
          if (grp == 0) {
            char *kr = p.pool + int64_t(page) * p.page_bytes + int64_t(slot & (P - 1)) * RB + part * 16;
            st16(kr, kp);
            st16(kr + int64_t(P) * RB, vp);
          }
#pragma unroll
          for (int h = 0; h < G; ++h) {
            const float d = row_sum<LPR>(qs[h].dot(kp)) * p.scale_log2;
            merge_state<VN>(m[h], ls[h], acc[h], d, 1.0f, cv);
          }
        }
        if (lane == 0) {
          if (has_cur) p.z[u] = znew;
          p.len_out[u] = (has_cur && !alpha) ? l + 1 : l;
          if (p.slot_index) p.slot_index[u] = has_cur ? slot : -1;
          if (flag) atomicOr(&p.ctrl->flags, flag);
          const int r0 = off / span;                  // range holding the unit's first slot
          p.meta[2 * u] = r0 + u;                     // its first partial record
          p.meta[2 * u + 1] = r - r0 + 1;             // number of pieces
        }
      }

      if (grp == 0) {
        if (start == 0 && owner) {     // the whole unit in one piece: final output
#pragma unroll
          for (int h = 0; h < G; ++h) {
            const float inv = ls[h] > 0.0f ? 1.0f / ls[h] : 0.0f;
#pragma unroll
            for (int e = 0; e < VN; ++e) acc[h][e] *= inv;
            char *op = static_cast<char *>(p.out) +
                       (int64_t(b * p.hq + g * G + h) * D + part * VN) * ES;
            st16(op, V::pack(acc[h]));
          }
        } else {                       // partial record r + u for the combine launch
#pragma unroll
          for (int h = 0; h < G; ++h) {
            float *rec = p.partials + (int64_t(r + u) * G + h) * REC;
            if (part == 0) {
              rec[0] = m[h];
              rec[1] = ls[h];
            }
#pragma unroll
            for (int e = 0; e < VN; ++e) rec[4 + part * VN + e] = acc[h][e];
          }
        }
      }
    }
  }
}

// Window grouping for the matrix-core decode: the mean of the segment's
// positions j - m + 1 .. j (m = min(j + 1, w); ring entries, then the new
// token from k, v with omega om) is formed in a vector layout -- lane owns
// elements E lane .. E lane + E - 1 -- and left in this wave's LDS area
// (fp32 key mean, then value mean) for the operand layout to pick up.
// Returns the window's omega sum.
template <int D>
__device__ __forceinline__ float window_mean_lds(const DecodeParams &p, int u, int j, float om,
                                                 float *lds) {
  constexpr int E = D / 64, RB = D * 2, kBatch = 4;
  const int lane = threadIdx.x & 63;
  const int W = p.win.window;
  const int m = min(j + 1, W);
  const char *ring = p.win.ring + int64_t(u) * W * 2 * RB + lane * E * 2;
  const float *wo = p.win.omega + int64_t(u) * W;
  float sk[E], sv[E], zs = 0.0f;
  {
    float kf[E], vf[E];
    load_e<2, E>(static_cast<const char *>(p.k) + int64_t(u) * RB + lane * E * 2, kf);
    load_e<2, E>(static_cast<const char *>(p.v) + int64_t(u) * RB + lane * E * 2, vf);
    if (lane == 0) kf[0] = 0.0f;   // k_t[0] <- 0
#pragma unroll
    for (int e = 0; e < E; ++e) {
      sk[e] = om * kf[e];
      sv[e] = om * vf[e];
    }
  }
  for (int i0 = j - m + 1; i0 < j; i0 += kBatch) {
    float kf[kBatch][E], vf[kBatch][E], wt[kBatch];
#pragma unroll
    for (int q = 0; q < kBatch; ++q) {
      const int i = i0 + q;
      const int ent = (i < j ? i : j - 1) % W;   // past the window: any entry, weight 0
      load_e<2, E>(ring + int64_t(ent) * 2 * RB, kf[q]);
      load_e<2, E>(ring + int64_t(ent) * 2 * RB + RB, vf[q]);
      wt[q] = i < j ? wo[ent] : 0.0f;
    }
#pragma unroll
    for (int q = 0; q < kBatch; ++q) {
#pragma unroll
      for (int e = 0; e < E; ++e) {
        sk[e] = fmaf(wt[q], kf[q][e], sk[e]);
        sv[e] = fmaf(wt[q], vf[q][e], sv[e]);
      }
      zs += wt[q];
    }
  }
  zs += om;
  const float inv = 1.0f / zs;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    lds[lane * E + e] = sk[e] * inv;
    lds[D + lane * E + e] = sv[e] * inv;
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  return zs;
}

// ---------------------------------------------------------------------------
// Grouped-query decode on matrix cores (bf16, G >= 4, pages of 32 slots).
//
// Same slot-space split, owner rule and partial records as decode_kernel;
// only the per-chunk arithmetic differs.  With G query heads per kv head the
// chunk work is G dot products and G weighted sums per cached row, too much
// for the vector ALUs at HBM speed, so both products run on
// v_mfma_f32_16x16x32_bf16 (query heads padded to 16):
//   scores  S^T[row][head] = K[row][:] . Q[head][:]   (A = K, B = Q^T)
//   values  O^T[dim][head] += V^T[dim][row] P^T[row][head]   (A = V^T, B = P^T)
// Key rows are assigned to the two 16-row score tiles interleaved (tile t,
// tile row m -> chunk row 8(m/4) + 4t + m%4) so that each lane ends up with
// the 8 consecutive rows 8q..8q+7 of one head -- exactly its slice of the
// P^T operand of the value product.  Value pages of such caches are stored
// transposed (V^T: d rows of page_size slots) so that slice of V^T is one
// 16-byte load.  P enters the value product rounded to bf16; its row sum is
// taken over the same rounded values.
//
// Chunks stream through LDS: each wave owns two chunk-sized LDS slots (keys,
// then V^T), filled by direct global-to-LDS transfers.  The wave copies a
// landed chunk into its operand registers and refills that slot with the
// chunk two ahead before computing on the registers, so two chunks (32 KB at
// d = 128) are in flight while one is consumed.  The ring takes 128 KB of LDS
// at d = 128, so one workgroup (one wave per SIMD) runs on a compute unit.
// Rows are stored with their 16-byte pieces XOR-permuted so that the operand
// reads of 16 consecutive lanes (16 rows at one column) hit distinct bank
// groups.
// ---------------------------------------------------------------------------
// Key row r of a chunk: 16-byte piece c sits at position c ^ key_perm(r).
template <int CPR>
__device__ __forceinline__ int key_perm(int r) {
  return CPR == 16 ? ((r & 3) | (((r >> 3) & 3) << 2)) : (((r >> 1) & 1) | (((r >> 3) & 3) << 1));
}
// V^T row r (64 bytes: 32 slots): piece c sits at position c ^ ((r >> 2) & 3).

template <int D>
constexpr int mfma_ring_bytes() { return kWaves * 2 * 2 * 32 * D * 2; }   // 2 slots per wave

// Occupancy: at d = 128 the chunk ring (128 KB) leaves room for one workgroup
// per compute unit (one wave per SIMD); at d = 64 two fit.
template <int D>
constexpr int mfma_decode_wg_per_cu() { return D == 128 ? 1 : 2; }

template <int D, int G, bool WIN, bool GRP>
__global__ __launch_bounds__(kThreads, mfma_decode_wg_per_cu<D>()) void decode_mfma_kernel(DecodeParams p) {
  constexpr int KS = D / 32;      // k-steps of the score product
  constexpr int NT = D / 16;      // 16-dim tiles of the value product
  constexpr int RB = D * 2;       // bytes per key row
  constexpr int CPR = RB / 16;    // 16-byte pieces per key row
  constexpr int CH = 32 * RB;     // bytes of a chunk's keys (and of its V^T)
  constexpr int NX = CH / 1024;   // 1-KB wave transfers per half chunk
  constexpr int REC = D + 4;      // partial record: m, l, -, -, acc[D]
  static_assert(G >= 4 && G <= 16, "query group");
  static_assert(CPR == 8 || CPR == 16, "head dim");

  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int s_wsum[kWaves];
  // The chunk ring: slot 0 and slot 1 of every wave in arrays of their own
  // (see the LDS transfer helpers).
  static_assert(mfma_ring_bytes<D>() == 2 * kWaves * 2 * CH, "ring layout");
  __shared__ __align__(16) unsigned char s_ring0[kWaves * 2 * CH], s_ring1[kWaves * 2 * CH];
  const int U = p.units;
  int *s_off = reinterpret_cast<int *>(smem);
  const int ng = GRP ? (U + p.slot_group - 1) / p.slot_group : U;   // slot-space table entries - 1
  const size_t win_lds_off = align_up(size_t(ng + 1) * 4, 16);   // windowed means, 2 D fp32 per wave
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 15, q = lane >> 4;      // MFMA column (head or dim) and k-group
  const int P = 1 << p.log2p;
  const int krow = 8 * (n >> 2) + (n & 3);     // this lane's key row in score tile 0 (+4 in tile 1)
  const uint4 zero4 = make_uint4(0, 0, 0, 0);

  constexpr int OVH = kMfmaUnitOverhead;
  const int S = build_slot_space<GRP, OVH>(p, s_off, s_wsum);
  const int nwaves = gridDim.x * kWaves;
  int span = (S + kRangesPerWave * nwaves - 1) / (kRangesPerWave * nwaves);
  if (p.split_tile > 0 && span > p.split_tile) span = p.split_tile;
  // Whole units when that balances: wave w takes units [w U / W, (w + 1) U / W)
  // in full if no wave's share then exceeds the equal slot share by more than
  // kWholeUnitSlack.  Split units cost this kernel a piece start, an owner
  // epilogue and a partial record each (measured: a 70B-shaped layer of
  // lengths 2048 +- 32 at 407-426 us per call against 345-348 us at 2048
  // exactly), so near-uniform lengths -- one compression ratio for every head
  // -- stream faster without them.  Grouped tables and forced split sizes keep
  // the equal-slot ranges.
  bool whole = false;
  if constexpr (!GRP) {
    if (p.split_tile == 0 && U >= nwaves) {
      int mx = 0;
      for (int w = threadIdx.x; w < nwaves; w += kThreads) {
        const int u0 = static_cast<int>(int64_t(w) * U / nwaves);
        const int u1 = static_cast<int>(int64_t(w + 1) * U / nwaves);
        mx = max(mx, s_off[u1] - s_off[u0]);
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) mx = max(mx, __shfl_xor(mx, o, 64));
      if (lane == 0) s_wsum[wave] = mx;
      __syncthreads();
      for (int w = 0; w < kWaves; ++w) mx = max(mx, s_wsum[w]);
      whole = int64_t(mx) * 100 <= int64_t(span) * (100 + kWholeUnitSlack);
    }
  }
  const int nranges = whole ? nwaves : (S + span - 1) / span;

  for (int r = blockIdx.x * kWaves + wave; r < nranges; r += nwaves) {
    const int wu0 = whole ? static_cast<int>(int64_t(r) * U / nwaves) : 0;
    int pos = whole ? s_off[wu0] : r * span;
    const int pos_end = whole ? s_off[static_cast<int>(int64_t(r + 1) * U / nwaves)] : min(pos + span, S);
    int off;
    for (int u = whole ? (off = pos, wu0) : unit_at<GRP, OVH>(p, s_off, pos, off); pos < pos_end;
         ++u, off = pos) {
      if constexpr (!GRP) off = s_off[u];
      const int n_u = GRP ? max(p.len_in[u], 1) + OVH : s_off[u + 1] - off;
      const int start = pos - off;
      const int stop = min(pos_end, off + n_u) - off;
      pos = off + stop;
      const bool owner = stop == n_u;
      const int l = p.len_in[u];
      const int b = u / p.hkv, g = u - b * p.hkv;
      const int64_t pt = int64_t(u) * p.maxpages;
      const int end = min(owner ? n_u - 1 : stop, n_u - OVH - 1);   // closed slots

      // Q^T operand: lane (n, q) holds Q[head n][32 ks + 8q .. +8]; heads >= G are 0.
      uint4 qb[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        qb[ks] = n < G ? ld16(static_cast<const char *>(p.q) +
                              (int64_t(b * p.hq + g * G + n) * D + ks * 32 + 8 * q) * 2)
                       : zero4;
      if (q == 0) qb[0].x &= 0xffff0000u;              // Algorithm 1: q_t[0] <- 0

      float m = neg_inf(), ls = 0.0f;
      f32x4_t acc[NT];
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

      // Score product of one chunk: lane (n, q) gets rows 8q .. 8q+7 of head n.
      auto scores = [&](const uint4 (&ka)[2][KS], float (&sv)[8]) {
        f32x4_t s0 = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f}, s1 = s0;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          s0 = mfma_16x16x32(ka[0][ks], qb[ks], s0);
          s1 = mfma_16x16x32(ka[1][ks], qb[ks], s1);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          sv[i] = s0[i];
          sv[4 + i] = s1[i];
        }
      };
      // Online softmax + value product of one chunk (rows with a bit set in vbits are valid).
      auto values = [&](const float (&sraw)[8], uint4 (&va)[NT], uint32_t vbits) {
        const uint32_t mine = (vbits >> (8 * q)) & 0xffu;   // rows 8q .. 8q+7
        float sv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) sv[j] = ((mine >> j) & 1u) ? sraw[j] * p.scale_log2 : neg_inf();
        float mc = sv[0];
#pragma unroll
        for (int j = 1; j < 8; ++j) mc = fmaxf(mc, sv[j]);
        mc = max_halves(max_rows16(mc));   // lane swaps, no LDS traffic
        const float mn = fmaxf(m, mc);
        if (vbits == 0u) return;
        const float f = fast_exp2(m - mn);
        ls *= f;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[nt] *= f;
        m = mn;
        uint32_t pw[4];
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          pw[w] = bf16_pair(fast_exp2(sv[2 * w] - mn), fast_exp2(sv[2 * w + 1] - mn));
          ls += __uint_as_float(pw[w] << 16) + __uint_as_float(pw[w] & 0xffff0000u);
        }
        const uint4 pb = make_uint4(pw[0], pw[1], pw[2], pw[3]);
        // Rows past the unit's length hold unwritten page memory: clear them in V^T.
        uint32_t keep[4];
#pragma unroll
        for (int w = 0; w < 4; ++w)
          keep[w] = (((mine >> (2 * w)) & 1u) ? 0x0000ffffu : 0u) |
                    (((mine >> (2 * w + 1)) & 1u) ? 0xffff0000u : 0u);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          va[nt].x &= keep[0];
          va[nt].y &= keep[1];
          va[nt].z &= keep[2];
          va[nt].w &= keep[3];
          acc[nt] = mfma_16x16x32(va[nt], pb, acc[nt]);
        }
      };

      // Owner inputs are issued before the stream so that they arrive while it runs:
      // k_t[0], q_t[0] of the deciding heads, z, the open slot's page, and the lane's
      // parts of the current key and value rows (as B operand and value tiles).
      float k0 = 0.0f, q0 = 0.0f, zold = 0.0f;
      int open_page = -1;
      uint4 kt[KS];
      uint16_t vt[NT];
      if (owner) {
        const int dg = p.decision_src ? 0 : g;   // head whose neurons decide for this unit
        k0 = load_elem<2>(p.k, int64_t(b * p.hkv + dg) * D);
        q0 = load_elem<2>(p.q, int64_t(b * p.hq + dg * G) * D);
        if (l > 0) {
          zold = p.z[u];
          open_page = p.ptab[pt + ((l - 1) >> p.log2p)];
        }
        const char *kr = static_cast<const char *>(p.k) + int64_t(u) * RB;
        const uint16_t *vr = reinterpret_cast<const uint16_t *>(static_cast<const char *>(p.v) +
                                                                int64_t(u) * RB);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) kt[ks] = ld16(kr + ks * 64 + q * 16);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) vt[nt] = vr[16 * nt + n];
      }

      const int c_last = end > start ? (end - 1) >> 5 : -1;   // the piece's last chunk
      // The owner's open slot: copied from the ring when its chunk streams by
      // (the slot's last 32 rows are its page), else read from its page below.
      const int so = (l - 1) & (P - 1);
      const int c_open = (owner && l > 0 && ((l - 1) >> 5) == c_last) ? c_last : -1;
      uint4 ko[KS];
      uint16_t vo[NT];
      if (end > start) {
        const int c0 = start >> 5, c1 = c_last;
        auto range_of = [&](int ch, int &rlo, int &rhi) {
          const int row0 = ch << 5;
          rlo = max(start, row0) - row0;
          rhi = min(end, row0 + 32) - row0;
        };
        // The whole chunk (one page: P == 32) is transferred; rows outside
        // [start, end) are page memory of this unit whose scores and values
        // the validity bits mask.  Every step issues the 2 NX transfers of
        // the chunk two ahead (switched off past the piece's last chunk).
        // Page-table entries of the piece's chunks, one per lane, 64 chunks per batch with the
        // next batch loaded one batch ahead: no chunk transfer waits on a table lookup.
        int cb = c0;
        int pcur = p.ptab[pt + min(c0 + lane, c1)];
        int pnxt = p.ptab[pt + min(c0 + 64 + lane, c1)];
        auto page_of = [&](int ch) -> int {
          if (ch - cb >= 64) {
            cb += 64;
            pcur = pnxt;
            pnxt = p.ptab[pt + min(cb + 64 + lane, c1)];
          }
          return __builtin_amdgcn_readlane(pcur, ch - cb);
        };
        auto ring_slot = [&](auto sl_c) -> unsigned char * {
          return (decltype(sl_c)::value ? s_ring1 : s_ring0) + wave * 2 * CH;
        };
        auto issue = [&](int ch, auto sl_c) {
          const bool on = ch <= c1;
          unsigned char *slot_k = ring_slot(sl_c), *slot_v = slot_k + CH;
          const char *pg = uniform_ptr(p.pool + int64_t(page_of(min(ch, c1))) * p.page_bytes);
#pragma unroll
          for (int i = 0; i < NX; ++i) {
            const int o = 1024 * i + 16 * lane, r = o / RB, c = (o % RB) / 16;
            dma16_s_nt(slot_k + 1024 * i, pg, uint32_t(r * RB + 16 * (c ^ key_perm<CPR>(r))), on);
          }
#pragma unroll
          for (int i = 0; i < NX; ++i) {
            const int r = 16 * i + (lane >> 2), c = lane & 3;
            dma16_s_nt(slot_v + 1024 * i, pg + CH, uint32_t(r * 64 + 16 * (c ^ ((r >> 2) & 3))), on);
          }
        };
        auto bits = [&](int ch) -> uint32_t {
          int rlo, rhi;
          range_of(ch, rlo, rhi);
          const uint32_t hi_mask = rhi >= 32 ? 0xffffffffu : ((1u << rhi) - 1u);
          return hi_mask & ~((1u << rlo) - 1u);
        };
        uint4 ka[2][KS], va[NT];
        issue(c0, std::integral_constant<int, 0>{});
        issue(c0 + 1, std::integral_constant<int, 1>{});
        auto step = [&](auto sl_c, int ch) {
          wait_vmcnt<2 * NX>();   // this chunk has landed; the next may be in flight
          wave_ring_sync();
          const unsigned char *ck = ring_slot(sl_c), *cv = ck + CH;
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            const int rr = krow + 4 * t;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
              ka[t][ks] = *reinterpret_cast<const uint4 *>(
                  ck + rr * RB + 16 * ((4 * ks + q) ^ key_perm<CPR>(rr)));
          }
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
            va[nt] = *reinterpret_cast<const uint4 *>(cv + (16 * nt + n) * 64 +
                                                      16 * (q ^ ((n >> 2) & 3)));
          if (ch == c_open) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
              ko[ks] = *reinterpret_cast<const uint4 *>(
                  ck + so * RB + 16 * ((4 * ks + q) ^ key_perm<CPR>(so)));
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
              vo[nt] = *reinterpret_cast<const uint16_t *>(
                  cv + (16 * nt + n) * 64 + 16 * ((so >> 3) ^ ((n >> 2) & 3)) + (so & 7) * 2);
          }
          wave_ring_sync();   // the slot's reads come before its refill
          issue(ch + 2, sl_c);
          if (ch > c1) return;   // past the piece's last chunk (odd count)
          float sraw[8];
          scores(ka, sraw);
          values(sraw, va, bits(ch));
        };
        // Pairs of steps, one per slot (a step past the last chunk only keeps
        // the transfer count in step).
        for (int ch = c0; ch <= c1; ch += 2) {
          step(std::integral_constant<int, 0>{}, ch);
          step(std::integral_constant<int, 1>{}, ch + 1);
        }
      }

      // Owner: the open slot copied from the ring above, else from its page.
      int seg_len = 0;
      if (owner) {
        if (WIN && l > 0) seg_len = p.win.seg_len[u];
        if (l > 0) {
          if (c_open < 0) {
            const char *pg = p.pool + int64_t(open_page) * p.page_bytes;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) ko[ks] = ld16(pg + int64_t(so) * RB + ks * 64 + q * 16);
            const uint16_t *vtp = reinterpret_cast<const uint16_t *>(pg + int64_t(P) * RB);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) vo[nt] = vtp[(16 * nt + n) * P + so];
          }
        } else {
#pragma unroll
          for (int ks = 0; ks < KS; ++ks) ko[ks] = zero4;
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) vo[nt] = 0;
        }
      }

      if (owner) {
        // Algorithm 1 for unit u (decision, importance, merge or append).
        const int alpha = (l > 0 && k0 > p.c) ? 1 : 0;
        float om;
        if (p.omega_src == 0) {
          om = sigmoid_floor(q0);
        } else if (p.omega_src == 1) {
          const int dg = p.decision_src ? 0 : g;
          float sum = 0.0f;
          for (int h = 0; h < G; ++h)
            sum += sigmoid_floor(load_elem<2>(p.q, int64_t(b * p.hq + dg * G + h) * D));
          om = fmaxf(sum / G, 0x1p-100f);
        } else {
          om = 1.0f;   // uniform weighting
        }
        int flag = 0, slot, page = open_page;
        bool has_cur = true;
        float znew;
        if (alpha) {
          slot = l - 1;
          znew = zold + om;
        } else {
          slot = l;
          znew = om;
          if (l >= p.max_slots) {
            has_cur = false;
            flag = FLAG_SLOTS_EXHAUSTED;
          } else if ((l & (P - 1)) == 0) {
            int pg = 0;
            if (lane == 0) {
              const unsigned long long x = atomicAdd(&p.ctrl->pages_used, 1ull);
              pg = x < static_cast<unsigned long long>(p.num_pages) ? static_cast<int>(x) : -1;
            }
            pg = __shfl(pg, 0, 64);
            if (pg < 0) {
              has_cur = false;
              flag = FLAG_POOL_EXHAUSTED;
            } else {
              page = pg;
              if (lane == 0) p.ptab[pt + (l >> p.log2p)] = pg;
            }
          }
        }
        if (q == 0) kt[0].x &= 0xffff0000u;     // Algorithm 1: k_t[0] <- 0
        // Window grouping: the open slot is the mean of its segment's last w tokens,
        // formed in this wave's LDS area.
        const bool windowed = WIN && alpha;
        const float *wmean = reinterpret_cast<const float *>(smem + win_lds_off) + wave * 2 * D;
        if (windowed)
          znew = window_mean_lds<D>(p, u, seg_len, om,
                                    reinterpret_cast<float *>(smem + win_lds_off) + wave * 2 * D);
        // Current key (lanes hold dims 32 ks + 8q .. +8) and value (dims 16 nt + n).
        uint4 kc[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          float kf[8], of[8];
          V16<2>::unpack(kt[ks], kf);
          V16<2>::unpack(ko[ks], of);
          if (windowed) {
            const float4 x0 = *reinterpret_cast<const float4 *>(wmean + 32 * ks + 8 * q);
            const float4 x1 = *reinterpret_cast<const float4 *>(wmean + 32 * ks + 8 * q + 4);
            kf[0] = x0.x; kf[1] = x0.y; kf[2] = x0.z; kf[3] = x0.w;
            kf[4] = x1.x; kf[5] = x1.y; kf[6] = x1.z; kf[7] = x1.w;
          } else if (alpha) {
#pragma unroll
            for (int e = 0; e < 8; ++e) kf[e] = (of[e] * zold + kf[e] * om) / znew;
          }
          kc[ks] = V16<2>::pack(kf);
        }
        uint16_t vc[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          float vf = __uint_as_float(uint32_t(vt[nt]) << 16);
          if (windowed) vf = wmean[D + 16 * nt + n];
          else if (alpha) vf = (__uint_as_float(uint32_t(vo[nt]) << 16) * zold + vf * om) / znew;
          vc[nt] = static_cast<uint16_t>(bf16_bits(vf));
        }
        if (WIN && has_cur) {   // the token joins its segment's window ring
          const int W = p.win.window, j = alpha ? seg_len : 0, ent = j % W;
          char *er = p.win.ring + (int64_t(u) * W + ent) * 2 * RB;
          if (n == 0) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) st16(er + ks * 64 + q * 16, kt[ks]);
          }
          if (q == 0) {
            uint16_t *ev = reinterpret_cast<uint16_t *>(er + RB);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) ev[16 * nt + n] = vt[nt];
          }
          if (lane == 0) {
            p.win.omega[int64_t(u) * W + ent] = om;
            p.win.seg_len[u] = j + 1;
          }
        }
        if (has_cur) {
          char *pg = p.pool + int64_t(page) * p.page_bytes;
          const int so = slot & (P - 1);
          if (n == 0) {
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) st16(pg + int64_t(so) * RB + ks * 64 + q * 16, kc[ks]);
          }
          if (q == 0) {
            uint16_t *vtp = reinterpret_cast<uint16_t *>(pg + int64_t(P) * RB);
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) vtp[(16 * nt + n) * P + so] = vc[nt];
          }
        }
        // Attend to the old open slot (kept on append) and the current slot:
        // a pseudo-chunk with them as rows 0 and 1.
        const bool old_valid = !alpha && l > 0;
        uint4 ka[2][KS], va[NT];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          ka[0][ks] = n == 0 ? ko[ks] : (n == 1 ? kc[ks] : zero4);
          ka[1][ks] = zero4;
        }
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          va[nt] = q == 0 ? make_uint4(uint32_t(vo[nt]) | (uint32_t(vc[nt]) << 16), 0, 0, 0) : zero4;
        float sraw[8];
        scores(ka, sraw);
        values(sraw, va, (old_valid ? 1u : 0u) | (has_cur ? 2u : 0u));
        if (lane == 0) {
          if (has_cur) p.z[u] = znew;
          p.len_out[u] = (has_cur && !alpha) ? l + 1 : l;
          if (p.slot_index) p.slot_index[u] = has_cur ? slot : -1;
          if (flag) atomicOr(&p.ctrl->flags, flag);
          const int r0 = whole ? r : off / span;
          p.meta[2 * u] = r0 + u;
          p.meta[2 * u + 1] = r - r0 + 1;
        }
      }

      ls += __shfl_xor(ls, 16, 64);
      ls += __shfl_xor(ls, 32, 64);
      if (n < G) {
        if (start == 0 && owner) {     // the whole unit in one piece: final output
          const float inv = ls > 0.0f ? 1.0f / ls : 0.0f;
          uint16_t *op = static_cast<uint16_t *>(p.out) + int64_t(b * p.hq + g * G + n) * D + 4 * q;
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) {
            const uint2 w = make_uint2(bf16_pair(acc[nt][0] * inv, acc[nt][1] * inv),
                                       bf16_pair(acc[nt][2] * inv, acc[nt][3] * inv));
            *reinterpret_cast<uint2 *>(op + 16 * nt) = w;
          }
        } else {                       // partial record r + u for the combine launch
          float *rec = p.partials + (int64_t(r + u) * G + n) * REC;
          if (q == 0) {
            rec[0] = m;
            rec[1] = ls;
          }
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
            *reinterpret_cast<float4 *>(rec + 4 + 16 * nt + 4 * q) =
                make_float4(acc[nt][0], acc[nt][1], acc[nt][2], acc[nt][3]);
        }
      }
    }
  }
}

// Combine the split-K partial records of units with more than one tile:
// o = sum_i 2^(m_i - M) acc_i / sum_i 2^(m_i - M) l_i.  One wave per
// (b, query head); lane i fetches record i's max and sum, then every lane
// accumulates its E dims over the records.  The launch also copies the
// step's post-update lengths back into the layer's current-lengths buffer
// (every unit's owner wrote len_out; this launch runs after all of them).
template <int ES, int D, int G>
__global__ __launch_bounds__(kThreads) void combine_kernel(DecodeParams p, int batch) {
  constexpr int REC = D + 4;
  constexpr int E = D / 64;
  {
    const int i = blockIdx.x * kThreads + threadIdx.x;
    if (i < p.units) p.len_in[i] = p.len_out[i];
  }
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int bh = blockIdx.x * kWaves + wave;
  if (bh >= batch * p.hq) return;
  const int b = bh / p.hq, h = bh - b * p.hq;
  const int g = h / G, hg = h - g * G;
  const int u = b * p.hkv + g;
  const int first = p.meta[2 * u], nt = p.meta[2 * u + 1];   // records first .. first+nt-1
  if (nt <= 1) return;
  if (nt <= 4) {
    // Few records (the usual case): every load is issued at once, one round trip.
    float mi[4], li[4], a[4][E];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      mi[i] = neg_inf();
      li[i] = 0.0f;
#pragma unroll
      for (int e = 0; e < E; ++e) a[i][e] = 0.0f;
      if (i < nt) {
        const float *rec = p.partials + (int64_t(first + i) * G + hg) * REC;
        mi[i] = rec[0];
        li[i] = rec[1];
#pragma unroll
        for (int e = 0; e < E; ++e) a[i][e] = rec[4 + lane * E + e];
      }
    }
    const float M = fmaxf(fmaxf(mi[0], mi[1]), fmaxf(mi[2], mi[3]));
    float L = 0.0f, A[E];
#pragma unroll
    for (int e = 0; e < E; ++e) A[e] = 0.0f;
    if (M != neg_inf()) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float w = mi[i] == neg_inf() ? 0.0f : fast_exp2(mi[i] - M);
        L = fmaf(w, li[i], L);
#pragma unroll
        for (int e = 0; e < E; ++e) A[e] = fmaf(w, a[i][e], A[e]);
      }
    }
    const float inv = L > 0.0f ? 1.0f / L : 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) A[e] *= inv;
    store_e<ES, E>(static_cast<char *>(p.out) + (int64_t(bh) * D + lane * E) * ES, A);
    return;
  }
  float L = 0.0f, A[E];
#pragma unroll
  for (int e = 0; e < E; ++e) A[e] = 0.0f;
  float M = neg_inf();
  for (int i0 = 0; i0 < nt; i0 += 64) {           // running max over chunks of 64 records
    const int i = i0 + lane;
    const float mi = i < nt ? p.partials[(int64_t(first + i) * G + hg) * REC] : neg_inf();
    float mc = mi;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mc = fmaxf(mc, __shfl_xor(mc, o, 64));
    const float mn = fmaxf(M, mc);
    if (mn == neg_inf()) continue;
    const float sc = fast_exp2(M - mn);
    L *= sc;
#pragma unroll
    for (int e = 0; e < E; ++e) A[e] *= sc;
    M = mn;
    const float wi = i < nt ? fast_exp2(mi - M) : 0.0f;
    const float li = i < nt ? p.partials[(int64_t(first + i) * G + hg) * REC + 1] : 0.0f;
    float lw = wi * li;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) lw += __shfl_xor(lw, o, 64);
    L += lw;
    const int cnt = min(64, nt - i0);
    int j = 0;
    for (; j + 4 <= cnt; j += 4) {
      float w4[4], a4[4][E];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        w4[q] = __shfl(wi, j + q, 64);
        const float *rec = p.partials + (int64_t(first + i0 + j + q) * G + hg) * REC + 4 + lane * E;
#pragma unroll
        for (int e = 0; e < E; ++e) a4[q][e] = rec[e];
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int e = 0; e < E; ++e) A[e] = fmaf(w4[q], a4[q][e], A[e]);
    }
    for (; j < cnt; ++j) {
      const float w = __shfl(wi, j, 64);
      const float *rec = p.partials + (int64_t(first + i0 + j) * G + hg) * REC + 4 + lane * E;
#pragma unroll
      for (int e = 0; e < E; ++e) A[e] = fmaf(w, rec[e], A[e]);
    }
  }
  const float inv = L > 0.0f ? 1.0f / L : 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) A[e] *= inv;
  store_e<ES, E>(static_cast<char *>(p.out) + (int64_t(bh) * D + lane * E) * ES, A);
}


// ---------------------------------------------------------------------------
// Prefill compactor.
// ---------------------------------------------------------------------------

__device__ __forceinline__ int prompt_len(const PrefillParams &p, int b, bool raise) {
  if (!p.prompt_lens) return p.n;
  int x = p.prompt_lens[b];
  if (x < 0 || x > p.n) {
    if (raise) atomicOr(&p.ctrl->flags, FLAG_BAD_LENGTH);
    x = x < 0 ? 0 : p.n;
  }
  return x;
}

// Launch-order helpers.  Workgroups are dispatched round-robin over the 8
// XCDs (workgroup i to XCD i mod 8); xcd_order maps the launch index to a
// logical one so that consecutive logical workgroups run on the same XCD (its
// L2), in dispatch order.  A bijection on [0, n) for any n.
__device__ __forceinline__ int xcd_order(int lin, int n) {
  const int q = n >> 3, r = n & 7, x = lin & 7, j = lin >> 3;
  return x < r ? x * (q + 1) + j : r * (q + 1) + (x - r) * q + j;
}

// Importance omega of token t of unit (b, dg) (Sec. 3.1: sigmoid of the first
// query neuron), per the configured source; floored at 2^-100.
template <int ES>
__device__ __forceinline__ float token_omega(const PrefillParams &p, int b, int t, int dg, int G) {
  if (p.omega_src == 0)
    return sigmoid_floor(load_elem<ES>(p.q, b * p.qs[0] + t * p.qs[1] + (dg * G) * p.qs[2]));
  if (p.omega_src == 1) {
    float sum = 0.0f;
    for (int h = 0; h < G; ++h)
      sum += sigmoid_floor(load_elem<ES>(p.q, b * p.qs[0] + t * p.qs[1] + (dg * G + h) * p.qs[2]));
    return fmaxf(sum / G, 0x1p-100f);
  }
  return 1.0f;   // uniform weighting
}

// Pass 1, one workgroup per unit (units in XCD order): decisions from the
// decision neuron k[0] (the first token always opens a slot), and per 64-token
// chunk the mask and count of segment starts; the unit length.  STAGE (prompt
// attention, window grouping) also stores every token's decision and
// importance for the passes that read them; the exact compaction reads only
// k[0] here and forms omega itself.  AUX is the neuron loads' cache
// policy: each load brings in the first 128-byte line of a key row, which the
// pages pass reads again; while those lines fit the last-level cache they are
// kept (default policy), otherwise they are streamed (nontemporal).
template <int ES, bool STAGE, int AUX>
__global__ __launch_bounds__(kThreads) void prefill_decide_kernel(PrefillParams p) {
  __shared__ int s_tot[kWaves];
  const int u = xcd_order(blockIdx.x, gridDim.x);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = u / p.hkv, g = u - b * p.hkv, G = p.hq / p.hkv;
  const int dg = p.decision_src ? 0 : g;   // head whose neurons decide for this unit
  const int nb = prompt_len(p, b, tid == 0);
  int total = 0;
  constexpr int kBatch = STAGE ? 8 : 16;   // tokens whose decision neurons are in flight per thread
  // Neurons by buffer loads with cache policy AUX: per batch and wave a
  // resource based at the wave's first token (SGPRs) and one lane offset
  // lane * token stride (below 2^31: the host bounds token strides), lanes past
  // the prompt switched off by an out-of-range offset -- no 64-bit address per
  // load and lane, so that every workgroup of a large layer is resident at once.
  const char *kb = static_cast<const char *>(p.k) + (b * p.ks[0] + dg * p.ks[2]) * ES;
  const char *qb = static_cast<const char *>(p.q) + (b * p.qs[0] + (dg * G) * p.qs[2]) * ES;
  const int64_t kst = p.ks[1] * ES, qst = p.qs[1] * ES;
  const uint32_t koff = lane * static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(kst)));
  const uint32_t qoff = lane * static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(qst)));
  auto neuron = [&](const char *base, int64_t st, uint32_t off, int tw) {
    const bool on = tw < p.n;   // wave-uniform
    const __amdgpu_buffer_rsrc_t rs = raw_rsrc(uniform_ptr(base + int64_t(on ? tw : 0) * st), on);
    const uint32_t vo = tw + lane < p.n ? off : kOutOfRange;
    if constexpr (ES == 2)
      return __uint_as_float(uint32_t(__builtin_amdgcn_raw_buffer_load_b16(rs, vo, 0, AUX)) << 16);
    else
      return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs, vo, 0, AUX));
  };
  for (int t00 = 0; t00 < p.n; t00 += kThreads * kBatch) {
    float k0[kBatch], q0[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int tw = t00 + j * kThreads + wave * 64;   // the wave's first token
      k0[j] = neuron(kb, kst, koff, tw);
      q0[j] = STAGE && p.omega_src == 0 ? neuron(qb, qst, qoff, tw) : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int t0 = t00 + j * kThreads;
      if (t0 < p.n) {   // (a wave-uniform condition)
      const int t = t0 + tid;
      int start = 0;
      if (t < p.n) {
        const bool valid = t < nb;
        const int a = (t > 0 && k0[j] > p.c) ? 1 : 0;
        if (STAGE) {
          const float om = p.omega_src == 0 ? sigmoid_floor(q0[j]) : token_omega<ES>(p, b, t, dg, G);
          p.alpha[int64_t(u) * p.max_prompt + t] = valid ? a : 1;
          p.omega[int64_t(u) * p.max_prompt + t] = om;
        }
        if (p.slot_index && !valid) p.slot_index[int64_t(u) * p.n + t] = -1;
        start = (valid && !a) ? 1 : 0;
      }
      const unsigned long long mask = __ballot(start);
      const int chunk = (t0 >> 6) + wave;
      if (lane == 0 && chunk * 64 < p.n) {
        p.count[int64_t(u) * p.prompt_chunks + chunk] = __popcll(mask);
        p.mask[int64_t(u) * p.prompt_chunks + chunk] = mask;
        total += __popcll(mask);
      }
      }
    }
  }
  if (lane == 0) s_tot[wave] = total;
  __syncthreads();
  if (tid == 0) {
    int l = 0;
    for (int w = 0; w < kWaves; ++w) l += s_tot[w];
    p.len[u] = l;
  }
}

// Pass 2 (also used by import), one workgroup: pages for every unit by an
// exclusive scan of ceil(l / P), contiguous per unit, from the bump pointer.
// The kernels that write the slots fill the page table.
__global__ __launch_bounds__(1024) void alloc_pages_kernel(int32_t *len, float *z,
                                                           int32_t *ptab, int32_t *page_base,
                                                           Control *ctrl, int64_t num_pages,
                                                           const int32_t *lengths_in,
                                                           const float *z_in, int32_t limit,
                                                           int units, int maxpages, int log2p) {
  __shared__ int s_wsum[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nthreads = blockDim.x;
  const int nw = nthreads / 64;
  const int per = (units + nthreads - 1) / nthreads;
  const int i0 = min(tid * per, units), i1 = min(i0 + per, units);
  const int P = 1 << log2p;
  const long long base = static_cast<long long>(ctrl->pages_used);
  int sum = 0, bad = 0;
  for (int i = i0; i < i1; ++i) {
    int l;
    if (lengths_in) {
      l = lengths_in[i];
      if (l < 0 || l > limit) {
        bad = 1;
        l = 0;
      }
      len[i] = l;
      z[i] = (l > 0) ? z_in[i] : 0.0f;
    } else {
      l = len[i];
      z[i] = 0.0f;
    }
    sum += (l + P - 1) >> log2p;
  }
  if (bad) atomicOr(&ctrl->flags, FLAG_BAD_LENGTH);
  int incl = sum;
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(incl, o, 64);
    if (lane >= o) incl += t;
  }
  if (lane == 63) s_wsum[wave] = incl;
  __syncthreads();
  long long run = incl - sum, total = 0;
  for (int w = 0; w < nw; ++w) {
    if (w < wave) run += s_wsum[w];
    total += s_wsum[w];
  }
  const bool fail = base + total > num_pages;
  for (int i = i0; i < i1; ++i) {
    const int l = len[i];
    const int np = (l + P - 1) >> log2p;
    if (fail) {
      page_base[i] = -1;
      len[i] = 0;
    } else {
      page_base[i] = static_cast<int>(base + run);   // the slot writers fill the page table
    }
    run += np;
  }
  __syncthreads();
  if (tid == 0) {
    if (fail) {
      atomicOr(&ctrl->flags, FLAG_POOL_EXHAUSTED);
      ctrl->alloc_count = 0;
    } else {
      ctrl->pages_used = static_cast<unsigned long long>(base + total);
      ctrl->alloc_base = base;
      ctrl->alloc_count = total;
    }
  }
}

#ifndef DMC_PF_ROWS
#define DMC_PF_ROWS 16
#endif
#ifndef DMC_PF_BUFFERS
#define DMC_PF_BUFFERS 1
#endif
constexpr int kPfRows = DMC_PF_ROWS;     // prompt rows per batch (each of K and V)
constexpr int kPfBuf = DMC_PF_BUFFERS;   // batches in a wave's register ring
static_assert(kPfRows >= 1 && kPfRows <= 32, "prompt rows per batch");
static_assert(kPfBuf >= 1 && kPfBuf <= 4, "ring depth");

// One lane's E elements of a prompt row as loaded (packed), unpacked at use.
template <int ES, int E>
struct RowBits {
  typedef typename std::conditional<(ES * E > 4), uint2, uint32_t>::type T;
  T w;
  // Nontemporal buffer load at rsrc + voff (lane) + soff (wave-uniform).
  __device__ __forceinline__ void load_nt(__amdgpu_buffer_rsrc_t rs, uint32_t voff, int soff) {
    if constexpr (ES == 2 && E == 2) {
      w = __builtin_amdgcn_raw_buffer_load_b32(rs, voff, soff, kNontemporal);
    } else if constexpr (ES == 2) {
      w = __builtin_amdgcn_raw_buffer_load_b16(rs, voff, soff, kNontemporal);
    } else if constexpr (E == 2) {
      typedef unsigned int u2_t __attribute__((ext_vector_type(2)));
      const u2_t x = __builtin_amdgcn_raw_buffer_load_b64(rs, voff, soff, kNontemporal);
      w = make_uint2(x.x, x.y);
    } else {
      w = __builtin_amdgcn_raw_buffer_load_b32(rs, voff, soff, kNontemporal);
    }
  }
  __device__ __forceinline__ void unpack(float *f) const {
    if constexpr (ES == 2 && E == 2) {
      f[0] = __uint_as_float(w << 16);
      f[1] = __uint_as_float(w & 0xffff0000u);
    } else if constexpr (ES == 2) {
      f[0] = __uint_as_float(w << 16);
    } else if constexpr (E == 2) {
      f[0] = __uint_as_float(w.x);
      f[1] = __uint_as_float(w.y);
    } else {
      f[0] = __uint_as_float(w);
    }
  }
};

// Position of the r-th set bit (r from 0) of m, which holds more than r bits.
__device__ __forceinline__ int select_bit(unsigned long long m, int r) {
  int pos = 0;
#pragma unroll
  for (int w = 32; w >= 1; w >>= 1) {
    const int c = __popcll(m & ((1ull << w) - 1ull));
    if (r >= c) {
      r -= c;
      m >>= w;
      pos += w;
    }
  }
  return pos;
}

__device__ __forceinline__ unsigned long long shfl64(unsigned long long x, int src) {
  const uint32_t lo = __shfl(static_cast<uint32_t>(x), src, 64);
  const uint32_t hi = __shfl(static_cast<uint32_t>(x >> 32), src, 64);
  return (static_cast<unsigned long long>(hi) << 32) | lo;
}

// Token that opens segment (slot) s of a unit, s < its length: the unit's
// start masks are read 64 chunks at a time (lane j: chunk j0 + j) and counted
// by a wave scan.  Returns `none` if the masks hold no such start.
__device__ __forceinline__ int start_token(const uint64_t *masks, int chunks, int s, int none) {
  const int lane = threadIdx.x & 63;
  int base = 0;
  for (int j0 = 0; j0 < chunks; j0 += 64) {
    const unsigned long long mk = j0 + lane < chunks ? masks[j0 + lane] : 0ull;
    const int c = __popcll(mk);
    int incl = c;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(incl, o, 64);
      if (lane >= o) incl += t;
    }
    const int tot = __shfl(incl, 63, 64);
    if (s < base + tot) {
      const int jl = __ffsll(static_cast<long long>(__ballot(base + incl > s))) - 1;
      const int before = base + __shfl(incl - c, jl, 64);
      return (j0 + jl) * 64 + select_bit(shfl64(mk, jl), s - before);
    }
    base += tot;
  }
  return none;
}

// Pass 3 (exact Algorithm 1), slot-aligned work items of about kItemTokens
// prompt tokens.  Unit u of length l is cut into items of S_u slots, S_u =
// l kItemTokens / n rounded up to a multiple of 32 (so an item of a highly
// compressed head spans few slots and one of an uncompressed head many, and
// every item reads about the same number of prompt rows).  32-slot alignment
// keeps every 32-slot page -- the transposed value pages of grouped-query
// caches included -- inside one item, written by one wave in whole rows, and
// no later pass touches it.  The item's tokens run from the start of its first
// slot's segment to the start of the segment after its last slot (the prompt
// end for the unit's last slot), located in the start masks of pass 1; each
// token is read once, by the item holding its segment.  A slot is the
// omega-weighted sum of its segment's keys (element 0 zeroed) and values over
// their omega sum, in fp32 -- the running mean Algorithm 1 holds at the
// segment's end; the unit's last segment gives z.  Omega comes from the first
// query neuron here.  With carry records enabled, the running sums of a
// segment that crosses a 32-token boundary t (t not a segment start) are
// stored as they stand before t, for the prompt-attention pass.  Waves map to
// (item k, unit u) with k outermost, in plain launch order, so every XCD gets
// a mix of all units and items.
//
// WIN (window grouping, Sec. 3.3; caches with transposed value pages): a
// slot is the omega-weighted mean of its segment's last min(w, length)
// tokens only, so a token counts when its segment ends within w tokens of it;
// the rows of the others are not read.  Omega comes from the staged
// importances, and the item holding the unit's last slot fills the unit's
// token ring from that segment's last tokens.  Writing the transposed value
// pages here replaces a separate page-transpose pass after the chunked
// window pass (Llama-2 70B GQA layer, w = 12: 1.92 -> 1.66 ms per call).
#ifndef DMC_PF_ITEM_TOKENS
#define DMC_PF_ITEM_TOKENS 128
#endif
constexpr int kItemTokens = DMC_PF_ITEM_TOKENS;

// Slots per work item of a unit with l slots from a prompt of n tokens.
__device__ __forceinline__ int item_slots(int l, int n) {
  const int64_t want = (int64_t(l) * kItemTokens + n - 1) / max(n, 1);
  return static_cast<int>(max<int64_t>(32, (want + 31) & ~int64_t(31)));
}

template <int ES, int D, bool VT, bool WIN>
__global__ __launch_bounds__(kThreads) void prefill_pages_kernel(PrefillParams p, int items) {
  constexpr int E = D / 64;         // elements per lane
  constexpr int RB = D * ES;        // bytes per row
  static_assert(!VT || ES == 2, "transposed value pages are bf16");
  static_assert(!WIN || VT, "row-layout caches with a window take prefill_window_kernel");
  __shared__ __align__(16) unsigned char s_vt[VT ? kWaves * 32 * RB : 16];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gw = blockIdx.x * kWaves + wave;
  const int k = gw / p.units;
  if (k >= items) return;
  const int u = gw - k * p.units, b = u / p.hkv, g = u - b * p.hkv;
  const int l = p.len[u];
  const int P = 1 << p.log2p;
  const int S = item_slots(l, p.n);
  const int s_lo = k * S;
  if (s_lo >= l) return;
  const int pb = p.page_base[u];
  if (pb < 0) return;
  const int s_hi = min(s_lo + S, l);
  const int nb = prompt_len(p, b, false);
  const int G = p.hq / p.hkv, dg = p.decision_src ? 0 : g;
  const uint64_t *um = p.mask + int64_t(u) * p.prompt_chunks;
  const int nch = (p.n + 63) >> 6;   // chunks written for this prompt
  // wave-uniform (the batch bounds below select SGPR row offsets)
  const int t_lo = __builtin_amdgcn_readfirstlane(start_token(um, nch, s_lo, nb));
  const int t_hi = __builtin_amdgcn_readfirstlane(s_hi < l ? start_token(um, nch, s_hi, nb) : nb);
  // Window grouping: lane j holds start-mask word c_base + j (re-read when a
  // batch's look-ahead passes the 64 words held), so that which rows a batch
  // needs is known before its loads are issued.
  const int W = WIN ? p.win.window : 0;
  int c_base = t_lo >> 6;
  unsigned long long held = 0;
  auto hold = [&](int c0) {
    c_base = c0;
    held = c0 + lane < nch ? um[c0 + lane] : 0ull;
  };
  if constexpr (WIN) hold(c_base);

  // page-table entries of the pages whose first slot is in the item
  const int64_t pt = int64_t(u) * p.maxpages;
  const int pg0 = (s_lo + P - 1) >> p.log2p, pg1 = (s_hi - 1) >> p.log2p;
  for (int i = pg0 + lane; i <= pg1; i += 64) p.ptab[pt + i] = pb + i;

  // Prompt rows are read by buffer loads: a resource based at the batch's
  // first row (SGPRs), a 32-bit row offset in an SGPR and one shared lane
  // offset -- a 64-bit address per row and lane took 64 of the kernel's
  // registers and halved its waves per SIMD.  Row offsets within a batch stay
  // below 2^31 bytes (the host bounds the row stride).
  const char *kbase = static_cast<const char *>(p.k) + (b * p.ks[0] + g * p.ks[2]) * ES;
  const char *vbase = static_cast<const char *>(p.v) + (b * p.vs[0] + g * p.vs[2]) * ES;
  const uint32_t lane_off = lane * E * ES;
  const int64_t kst = p.ks[1] * ES, vst = p.vs[1] * ES;
  const int kst32 = __builtin_amdgcn_readfirstlane(static_cast<int>(kst));
  const int vst32 = __builtin_amdgcn_readfirstlane(static_cast<int>(vst));
  unsigned char *stage = s_vt + (VT ? wave * 32 * RB : 0);
  // Byte offset of element e of staging row r: rows of RB bytes, unpadded (32 KB per
  // workgroup, so that five fit a compute unit), with the 4-byte word index XORed by
  // 8 (r / 8 mod 4).  A row write (64 lanes, consecutive words) and a column gather
  // (lanes over 16 elements x 4 row groups) then touch distinct banks.
  auto stage_at = [&](int r, int e) {
    const int byte = 2 * e;
    return r * RB + ((((byte >> 2) ^ (8 * ((r >> 3) & 3))) << 2) | (byte & 3));
  };
  int s = s_lo;
  int a_cur = t_lo;   // first token of slot s
  float ak[E], av[E], zs = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) ak[e] = av[e] = 0.0f;

  // The value page of grouped-query caches, staged as 32 rows in LDS, goes out
  // as V^T: lane (dim, quarter) gathers 8 slots of one dim -- conflict-free
  // thanks to the swizzle -- and stores them as one 16-byte piece.  The loop is
  // not unrolled: unrolled, its 64 reads in flight took 21 more VGPRs.
  auto write_vt_page = [&](char *vtp) {
    if constexpr (VT) {
      wave_lds_sync();
#pragma unroll 1
      for (int i = 0; i < D * 4 / 64; ++i) {
        const int pc = i * 64 + lane, dim = pc >> 2, qq = pc & 3;
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          w[j] = uint32_t(*reinterpret_cast<const uint16_t *>(stage + stage_at(8 * qq + 2 * j, dim))) |
                 (uint32_t(*reinterpret_cast<const uint16_t *>(stage + stage_at(8 * qq + 2 * j + 1, dim)))
                  << 16);
        __builtin_nontemporal_store(u32x4{w[0], w[1], w[2], w[3]},
                                    reinterpret_cast<u32x4 *>(vtp + dim * 64 + qq * 16));
      }
      wave_lds_sync();   // the staging rows are read before they are refilled
    }
  };
  auto flush = [&]() {   // slot s = sums / zs
    const float inv = 1.0f / zs;
    float kq[E], vq[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      kq[e] = ak[e] * inv;
      vq[e] = av[e] * inv;
    }
    const int row = s & (P - 1);
    char *pg = p.pool + int64_t(pb + (s >> p.log2p)) * p.page_bytes;
    store_e_nt<ES, E>(pg + int64_t(row) * RB + lane * E * ES, kq);
    if constexpr (VT) {
      store_e<ES, E>(reinterpret_cast<char *>(stage + stage_at(row, lane * E)), vq);
      if (row == 31 || s == s_hi - 1) write_vt_page(pg + 32 * RB);
    } else {
      store_e_nt<ES, E>(pg + int64_t(P) * RB + int64_t(row) * RB + lane * E * ES, vq);
    }
  };

  // Batches of kPfRows tokens stream through a ring of kPfBuf register
  // buffers: kPfBuf - 1 batches are in flight while one is consumed.  A batch
  // carries its K and V rows (packed), the lane's first query neuron (lane j:
  // token t2 + j) and the start-mask words that cover it.
  struct Batch {
    RowBits<ES, E> kr[kPfRows], vr[kPfRows];
    uint32_t q0;
    unsigned long long m0, m1;
  };
  const int nbat = (t_hi - t_lo + kPfRows - 1) / kPfRows;
  const bool lead_q0 = p.omega_src == 0;
  auto issue = [&](int bi, Batch &bt) {
    const int t2 = t_lo + bi * kPfRows, cnt = min(kPfRows, t_hi - t2);
    uint32_t need = ~0u;   // rows the batch needs (bit j: token t2 + j)
    if constexpr (WIN) {
      // Token t is needed when its segment ends within W tokens: a start in
      // (t, t + W], or the prompt end nb <= t + W.
      if (min((t2 + cnt - 1 + W) >> 6, nch - 1) >= c_base + 64) hold(t2 >> 6);
      const int t = t2 + lane, c = (t + 1) >> 6, sh = (t + 1) & 63;
      const unsigned long long w0 = shfl64(held, min(c - c_base, 63));
      const unsigned long long w1 = shfl64(held, min(c + 1 - c_base, 63));
      const unsigned long long ahead = sh ? (w0 >> sh) | (w1 << (64 - sh)) : w0;   // bit i: start t + 1 + i
      const unsigned long long wm = W >= 64 ? ~0ull : ((1ull << W) - 1ull);
      need = static_cast<uint32_t>(__ballot(lane < cnt && ((ahead & wm) != 0 || t + W >= nb)));
      const int c2 = t2 >> 6;
      bt.m0 = shfl64(held, c2 - c_base);
      bt.m1 = shfl64(held, min(c2 + 1 - c_base, 63));
      if (c2 + 1 >= nch) bt.m1 = 0ull;
    }
    // a row that is not needed is not read (its resource is switched off)
    const char *kb2 = uniform_ptr(kbase + t2 * kst), *vb2 = uniform_ptr(vbase + t2 * vst);
#pragma unroll
    for (int j = 0; j < kPfRows; ++j) {
      const int jj = min(j, cnt - 1);
      const bool on = !WIN || ((need >> jj) & 1u);
      bt.kr[j].load_nt(raw_rsrc(kb2, on), lane_off, jj * kst32);   // prompt rows are read once
      bt.vr[j].load_nt(raw_rsrc(vb2, on), lane_off, jj * vst32);
    }
    bt.q0 = 0;
    if constexpr (WIN) {
      // staged importances of the needed tokens (0 for the others)
      if (lane < cnt && ((need >> lane) & 1u))
        bt.q0 = __float_as_uint(p.omega[int64_t(u) * p.max_prompt + t2 + lane]);
      return;
    }
    if (lead_q0 && lane < cnt) {
      const int64_t qi = b * p.qs[0] + int64_t(t2 + lane) * p.qs[1] + (dg * G) * p.qs[2];
      bt.q0 = ES == 2 ? uint32_t(static_cast<const uint16_t *>(p.q)[qi]) << 16
                      : __float_as_uint(static_cast<const float *>(p.q)[qi]);
    }
    const int c2 = t2 >> 6;
    bt.m0 = um[c2];
    bt.m1 = ((t2 & 63) + kPfRows > 64 && c2 + 1 < nch) ? um[c2 + 1] : 0ull;
  };
  auto consume = [&](int bi, const Batch &bt) {
    const int t2 = t_lo + bi * kPfRows, cnt = min(kPfRows, t_hi - t2);
    // segment starts among the batch's tokens (bit j), the item's first token
    // (the start of slot s_lo) not counted
    const int sh = t2 & 63;
    unsigned long long w = bt.m0 >> sh;
    if (sh + kPfRows > 64) w |= bt.m1 << (64 - sh);
    uint32_t sb = static_cast<uint32_t>(w) & (kPfRows == 32 ? ~0u : ((1u << kPfRows) - 1u));
    if (t2 == t_lo) sb &= ~1u;
    const float om_lane = lane >= cnt ? 0.0f
                          : WIN     ? __uint_as_float(bt.q0)
                          : lead_q0 ? sigmoid_floor(__uint_as_float(bt.q0))
                                    : token_omega<ES>(p, b, t2 + lane, dg, G);
    if (p.slot_index && lane < cnt)
      p.slot_index[int64_t(u) * p.n + t2 + lane] = s + __popc(sb & ((2u << lane) - 1u));
#pragma unroll
    for (int j = 0; j < kPfRows; ++j) {
      if (j < cnt) {
        const int tj = t2 + j;
        if ((sb >> j) & 1u) {   // the next slot's segment opens
          flush();
          ++s;
          a_cur = tj;
          zs = 0.0f;
#pragma unroll
          for (int e = 0; e < E; ++e) ak[e] = av[e] = 0.0f;
        } else if (p.carry && tj != t_lo && (tj & 31) == 0) {
          float *cr = p.carry + (int64_t(u) * p.carry_blocks + (tj >> 5)) * carry_stride(D);
#pragma unroll
          for (int e = 0; e < E; ++e) {
            cr[lane * E + e] = ak[e];
            cr[D + lane * E + e] = av[e];
          }
          if (lane == 0) cr[2 * D] = zs;
        }
        const float om = __shfl(om_lane, j, 64);
        float kf[E], vf[E];
        bt.kr[j].unpack(kf);
        bt.vr[j].unpack(vf);
        if (lane == 0) kf[0] = 0.0f;   // k_t[0] <- 0
#pragma unroll
        for (int e = 0; e < E; ++e) {
          ak[e] = fmaf(om, kf[e], ak[e]);
          av[e] = fmaf(om, vf[e], av[e]);
        }
        zs += om;
      }
    }
  };
  Batch ring[kPfBuf];
#pragma unroll
  for (int j = 0; j < kPfBuf - 1; ++j)
    if (j < nbat) issue(j, ring[j]);
  for (int bi = 0; bi < nbat; bi += kPfBuf) {
#pragma unroll
    for (int j = 0; j < kPfBuf; ++j) {
      if (bi + j < nbat) {
        if (bi + j + kPfBuf - 1 < nbat) issue(bi + j + kPfBuf - 1, ring[(j + kPfBuf - 1) % kPfBuf]);
        consume(bi + j, ring[j]);
      }
    }
  }
  flush();   // slot s_hi - 1
  if (s_hi == l && lane == 0) p.z[u] = zs;   // the unit's last segment
  if constexpr (WIN) {
    if (s_hi == l) {
      // The unit's open segment (slot l - 1, from token a_cur): its last
      // min(W, length) tokens fill the token ring, position i of the segment
      // in entry i mod W, with their importances.  These (at most W) rows are
      // read again here rather than kept through the loop above.
      const int len = nb - a_cur;
      constexpr int R = 8;
      for (int i0 = max(0, len - W); i0 < len; i0 += R) {
        const int cnt = min(R, len - i0);
        const __amdgpu_buffer_rsrc_t krs = raw_rsrc(uniform_ptr(kbase + int64_t(a_cur + i0) * kst));
        const __amdgpu_buffer_rsrc_t vrs = raw_rsrc(uniform_ptr(vbase + int64_t(a_cur + i0) * vst));
        RowBits<ES, E> kr[R], vr[R];
#pragma unroll
        for (int j = 0; j < R; ++j) {
          const int jj = min(j, cnt - 1);
          kr[j].load_nt(krs, lane_off, jj * kst32);
          vr[j].load_nt(vrs, lane_off, jj * vst32);
        }
        const float om_lane = lane < cnt ? p.omega[int64_t(u) * p.max_prompt + a_cur + i0 + lane] : 0.0f;
#pragma unroll
        for (int j = 0; j < R; ++j) {
          if (j < cnt) {
            const int ent = (i0 + j) % W;
            float kf[E], vf[E];
            kr[j].unpack(kf);
            vr[j].unpack(vf);
            if (lane == 0) kf[0] = 0.0f;   // k_t[0] <- 0
            char *er = p.win.ring + (int64_t(u) * W + ent) * 2 * RB + lane * E * ES;
            store_e<ES, E>(er, kf);
            store_e<ES, E>(er + RB, vf);
            const float om = __shfl(om_lane, j, 64);
            if (lane == 0) p.win.omega[int64_t(u) * W + ent] = om;
          }
        }
      }
      if (lane == 0) p.win.seg_len[u] = len;
    }
  }
}

// Pass 3 with window grouping (Sec. 3.3) for caches whose value pages hold
// rows, one wave per (unit, 64-token chunk): every segment whose first token lies in the chunk becomes the
// omega-weighted mean of its last min(w, length) tokens -- the state the
// windowed partial accumulation reaches at the segment's end.  Only those
// tokens are read: the wave lists, in order, the tokens of its segments that
// lie within w of their segment's end (at most 64 in the chunk, plus up to w
// of the last segment past the chunk end) and streams them in batches,
// flushing a slot whenever the segment changes.  The wave holding the
// unit's last segment also fills the unit's token ring (position j of the
// segment in entry j mod w) and writes z and the open segment's length.
// Slot indices of every token come from the segment-start mask.
template <int ES, int D>
__global__ __launch_bounds__(kThreads) void prefill_window_kernel(PrefillParams p) {
  constexpr int E = D / 64;  // elements per lane
  constexpr int RB = D * ES;
  constexpr int kRows = 8;   // token rows in flight per wave
  __shared__ int s_list[kWaves][64 + kMaxWindow];
  const int u = blockIdx.y, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ch = blockIdx.x * kWaves + wave;
  const int tlo = ch * 64;
  if (tlo >= p.n) return;
  const int pb = p.page_base[u];
  if (pb < 0) return;
  const int b = u / p.hkv, g = u - b * p.hkv;
  const int nb = prompt_len(p, b, false);
  if (tlo >= nb) return;
  const uint8_t *al = p.alpha + int64_t(u) * p.max_prompt;
  const float *om = p.omega + int64_t(u) * p.max_prompt;
  auto starts = [&](int wb) -> unsigned long long {
    const int t = wb + lane;
    return __ballot(t < nb && al[t] == 0);
  };
  const unsigned long long m0 = starts(tlo);
  if (m0 == 0) return;
  int before = 0;
  for (int j = lane; j < ch; j += 64) before += p.count[int64_t(u) * p.prompt_chunks + j];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) before += __shfl_xor(before, o, 64);
  const int t0 = tlo + __ffsll(static_cast<long long>(m0)) - 1;
  int t_stop = nb;
  for (int wb = tlo + 64; wb < nb; wb += 64) {
    const unsigned long long mk = starts(wb);
    if (mk) {
      t_stop = wb + __ffsll(static_cast<long long>(mk)) - 1;
      break;
    }
  }
  const int W = p.win.window;
  const int nseg = __popcll(m0);
  const int a_last = tlo + 63 - __clzll(static_cast<long long>(m0));   // start of the last segment
  // Segment of token t in [t0, t_stop) (relative to `before`).
  auto seg_of = [&](int t) {
    const int rel = t - tlo;
    return rel < 64 ? __popcll(m0 & (rel == 63 ? ~0ull : ((2ull << rel) - 1ull))) - 1 : nseg - 1;
  };

  // Slot index of every token of the chunk's segments.
  if (p.slot_index) {
    for (int tb = t0; tb < t_stop; tb += 64) {
      const int t = tb + lane;
      if (t < t_stop) p.slot_index[int64_t(u) * p.n + t] = before + seg_of(t);
    }
  }

  // Token list: chunk tokens within w of their segment's end, then the last
  // segment's tokens past the chunk end that are within w of t_stop.
  int total;
  {
    const int t = tlo + lane;
    const unsigned long long later = m0 & (lane == 63 ? 0ull : (~0ull << (lane + 1)));
    const int seg_end = later ? tlo + __ffsll(static_cast<long long>(later)) - 1 : t_stop;
    const bool keep = t >= t0 && t < t_stop && t >= seg_end - W;
    const unsigned long long mk = __ballot(keep);
    if (keep) s_list[wave][__popcll(mk & ((1ull << lane) - 1ull))] = t;
    const int nin = __popcll(mk);
    const int tail0 = max(tlo + 64, t_stop - W);
    const int ntail = max(0, t_stop - tail0);   // <= W
    for (int i = lane; i < ntail; i += 64) s_list[wave][nin + i] = tail0 + i;
    total = nin + ntail;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  }

  const int P = 1 << p.log2p;
  const char *kbase = static_cast<const char *>(p.k) + (b * p.ks[0] + g * p.ks[2] + lane * E) * ES;
  const char *vbase = static_cast<const char *>(p.v) + (b * p.vs[0] + g * p.vs[2] + lane * E) * ES;
  const int64_t kst = p.ks[1] * ES, vst = p.vs[1] * ES;
  const bool last_unit_seg = t_stop >= nb;   // the chunk's last segment is the unit's last
  char *ring = p.win.ring + int64_t(u) * W * 2 * RB + lane * E * ES;
  float *ring_w = p.win.omega + int64_t(u) * W;
  int s = -1;
  float ak[E], av[E], zs = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) ak[e] = av[e] = 0.0f;
  auto flush = [&]() {   // write slot before + s = sums / zs
    const int sl = before + s;
    const float inv = 1.0f / zs;
    float kq[E], vq[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      kq[e] = ak[e] * inv;
      vq[e] = av[e] * inv;
    }
    char *row = p.pool + int64_t(pb + (sl >> p.log2p)) * p.page_bytes + int64_t(sl & (P - 1)) * RB +
                lane * E * ES;
    store_e_nt<ES, E>(row, kq);
    store_e_nt<ES, E>(row + int64_t(P) * RB, vq);
    if (lane == 0 && (sl & (P - 1)) == 0)
      p.ptab[int64_t(u) * p.maxpages + (sl >> p.log2p)] = pb + (sl >> p.log2p);
  };
  for (int i0 = 0; i0 < total; i0 += kRows) {
    const int cnt = min(kRows, total - i0);
    int tk[kRows];
    float kk[kRows][E], vv[kRows][E], ww[kRows];
#pragma unroll
    for (int j = 0; j < kRows; ++j) {
      tk[j] = s_list[wave][i0 + min(j, cnt - 1)];
      load_e_nt<ES, E>(kbase + tk[j] * kst, kk[j]);   // prompt rows are read once
      load_e_nt<ES, E>(vbase + tk[j] * vst, vv[j]);
      ww[j] = om[tk[j]];
    }
#pragma unroll
    for (int j = 0; j < kRows; ++j) {
      if (j < cnt) {
        const int sj = seg_of(tk[j]);
        if (sj != s) {   // the next segment's window begins
          if (s >= 0) flush();
          s = sj;
          zs = 0.0f;
#pragma unroll
          for (int e = 0; e < E; ++e) ak[e] = av[e] = 0.0f;
        }
        if (lane == 0) kk[j][0] = 0.0f;   // k_t[0] <- 0
#pragma unroll
        for (int e = 0; e < E; ++e) {
          ak[e] = fmaf(ww[j], kk[j][e], ak[e]);
          av[e] = fmaf(ww[j], vv[j][e], av[e]);
        }
        zs += ww[j];
        if (last_unit_seg && sj == nseg - 1) {   // the unit's open segment: fill its ring
          const int ent = (tk[j] - a_last) % W;
          store_e<ES, E>(ring + int64_t(ent) * 2 * RB, kk[j]);
          store_e<ES, E>(ring + int64_t(ent) * 2 * RB + RB, vv[j]);
          if (lane == 0) ring_w[ent] = ww[j];
        }
      }
    }
  }
  flush();
  if (last_unit_seg && lane == 0) {
    p.z[u] = zs;
    p.win.seg_len[u] = t_stop - a_last;
  }
}

// ---------------------------------------------------------------------------
// Dense <-> paged copies (import / export) and small utilities.
// ---------------------------------------------------------------------------
constexpr int kDenseRows = 16;

template <int ES, int D>
__global__ __launch_bounds__(kThreads) void import_kernel(DenseParams p) {
  constexpr int RB = D * ES, CPR = RB / 16;
  const int u = blockIdx.y;
  const int pb = p.page_base[u];
  if (pb < 0) return;
  const int l = p.len[u];
  const int P = 1 << p.log2p;
  for (int idx = threadIdx.x; idx < kDenseRows * CPR; idx += kThreads) {
    const int r = idx / CPR, c = idx - r * CPR;
    const int s = blockIdx.x * kDenseRows + r;
    if (s >= l) continue;
    const int64_t src = (int64_t(u) * p.dense_slots + s) * RB + c * 16;
    char *dst = p.pool + int64_t(pb + (s >> p.log2p)) * p.page_bytes + int64_t(s & (P - 1)) * RB + c * 16;
    if (c == 0 && (s & (P - 1)) == 0) p.ptab[int64_t(u) * p.maxpages + (s >> p.log2p)] = pb + (s >> p.log2p);
    st16(dst, ld16(static_cast<const char *>(p.kd) + src));
    st16(dst + int64_t(P) * RB, ld16(static_cast<const char *>(p.vd) + src));
  }
}

template <int ES, int D, bool VT>
__global__ __launch_bounds__(kThreads) void export_kernel(DenseParams p) {
  constexpr int RB = D * ES, CPR = RB / 16;
  const int u = blockIdx.y;
  const int l = p.len[u];
  const int P = 1 << p.log2p;
  if (blockIdx.x == 0 && threadIdx.x == 0) p.z_out[u] = p.z[u];
  for (int idx = threadIdx.x; idx < kDenseRows * CPR; idx += kThreads) {
    const int r = idx / CPR, c = idx - r * CPR;
    const int s = blockIdx.x * kDenseRows + r;
    if (s >= p.dense_slots) continue;
    const int64_t dst = (int64_t(u) * p.dense_slots + s) * RB + c * 16;
    uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
    if (s < l) {
      const int page = p.ptab[int64_t(u) * p.maxpages + (s >> p.log2p)];
      const char *src = p.pool + int64_t(page) * p.page_bytes + int64_t(s & (P - 1)) * RB + c * 16;
      kv = ld16(src);
      if constexpr (VT) {
        const uint16_t *vt = reinterpret_cast<const uint16_t *>(p.pool + int64_t(page) * p.page_bytes +
                                                                int64_t(P) * RB);
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          w[j] = uint32_t(vt[(c * 8 + 2 * j) * P + (s & (P - 1))]) |
                 (uint32_t(vt[(c * 8 + 2 * j + 1) * P + (s & (P - 1))]) << 16);
        vv = make_uint4(w[0], w[1], w[2], w[3]);
      } else {
        vv = ld16(src + int64_t(P) * RB);
      }
    }
    st16(static_cast<char *>(p.kd) + dst, kv);
    st16(static_cast<char *>(p.vd) + dst, vv);
  }
}

// Value pages of matrix-core caches (32-slot pages) are stored transposed
// ([d][32] bf16).  Prefill and import write rows ([32][d]); this pass turns
// the pages the last allocation handed out into the transposed form, one
// page per workgroup iteration: the whole page is read into LDS (row stride
// padded against bank conflicts) before any of it is overwritten.
template <int D>
__global__ __launch_bounds__(kThreads) void transpose_v_pages_kernel(char *pool, int64_t page_bytes,
                                                                     const Control *ctrl) {
  constexpr int RB = D * 2;
  constexpr int LDW = D + 2;                  // padded LDS row, in bf16 elements
  constexpr int CHUNKS = 32 * RB / 16;        // 16-byte pieces of a page's value rows
  constexpr int PER = (CHUNKS + kThreads - 1) / kThreads;
  __shared__ uint16_t tile[32 * LDW];
  const long long base = ctrl->alloc_base, count = ctrl->alloc_count;
  for (long long job = blockIdx.x; job < count; job += gridDim.x) {
    char *vreg = pool + (base + job) * page_bytes + 32 * RB;
    uint4 rows[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int idx = k * kThreads + threadIdx.x;
      if (idx < CHUNKS) rows[k] = ld16(vreg + int64_t(idx) * 16);
    }
    __syncthreads();   // every reader of the previous page's tile is done
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int idx = k * kThreads + threadIdx.x;
      if (idx < CHUNKS) {
        const int r = idx / (RB / 16), c = (idx % (RB / 16)) * 8;
        const uint32_t w[4] = {rows[k].x, rows[k].y, rows[k].z, rows[k].w};
#pragma unroll
        for (int j = 0; j < 8; ++j) tile[r * LDW + c + j] = static_cast<uint16_t>(w[j >> 1] >> (16 * (j & 1)));
      }
    }
    __syncthreads();   // the page is fully in LDS before it is overwritten
    // V^T[dim][8g .. 8g+7] for every dim and 8-row group g: 16-byte stores
    for (int idx = threadIdx.x; idx < D * 4; idx += kThreads) {
      const int dim = idx >> 2, g8 = (idx & 3) * 8;
      uint32_t w[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        w[j] = uint32_t(tile[(g8 + 2 * j) * LDW + dim]) | (uint32_t(tile[(g8 + 2 * j + 1) * LDW + dim]) << 16);
      st16(vreg + (int64_t(dim) * 32 + g8) * 2, make_uint4(w[0], w[1], w[2], w[3]));
    }
  }
}

__global__ void fill_i32_kernel(int32_t *p, int32_t v, size_t n) {
  for (size_t i = blockIdx.x * size_t(blockDim.x) + threadIdx.x; i < n; i += size_t(gridDim.x) * blockDim.x)
    p[i] = v;
}

__global__ void zero_u8_kernel(uint8_t *p, size_t n) {
  for (size_t i = blockIdx.x * size_t(blockDim.x) + threadIdx.x; i < n; i += size_t(gridDim.x) * blockDim.x)
    p[i] = 0;
}

__global__ void copy_i32_kernel(int32_t *d, const int32_t *s, size_t n) {
  for (size_t i = blockIdx.x * size_t(blockDim.x) + threadIdx.x; i < n; i += size_t(gridDim.x) * blockDim.x)
    d[i] = s[i];
}

int grid_for(size_t n) {
  const size_t g = (n + kThreads - 1) / kThreads;
  return static_cast<int>(g < 4096 ? (g > 0 ? g : 1) : 4096);
}

template <int D>
hipError_t launch_transpose(char *pool, int64_t page_bytes, const Control *ctrl, hipStream_t s) {
  hipLaunchKernelGGL((transpose_v_pages_kernel<D>), dim3(2048), dim3(kThreads), 0, s, pool,
                     page_bytes, ctrl);
  return hipGetLastError();
}

template <int ES, int D, int G, bool WIN, bool GRP>
void launch_decode_kernel(const DecodeParams &p, int grid, bool vt, size_t lds, hipStream_t s) {
  if constexpr (ES == 2 && G >= 4) {
    if (vt) {
      hipLaunchKernelGGL((decode_mfma_kernel<D, G, WIN, GRP>), dim3(grid), dim3(kThreads), lds, s, p);
      return;
    }
  }
  // grid counts workgroups of kThreads; the vector kernel packs the same waves
  // into workgroups of valu_decode_threads<ES, G>()
  constexpr int NT = valu_decode_threads<ES, G>();
  const int vgrid = std::max(1, grid / (NT / kThreads));
  hipLaunchKernelGGL((decode_kernel<ES, D, G, WIN, GRP>), dim3(vgrid), dim3(NT), lds, s, p);
}

template <int ES, int D, int G>
hipError_t decode_impl(const DecodeParams &p, int grid, bool vt, hipStream_t s) {
  const size_t lds = decode_lds_bytes((p.units + p.slot_group - 1) / p.slot_group + 1, G, D,
                                      p.win.window > 0);
  if (vt && !(ES == 2 && G >= 4)) return hipErrorInvalidValue;
  // The matrix-core kernel adds its chunk ring to the LDS of a workgroup.  When
  // two such workgroups do not fit a compute unit (always at d = 128), the grid
  // is halved so that every workgroup is resident at once.
  constexpr size_t kLdsPerCu = 160 * 1024;
  if (vt && 2 * (lds + mfma_ring_bytes<D>() + 64) > kLdsPerCu && grid > 1)
    grid /= 2;
  // grouped slot-space tables are built for exact (window-free) caches only
  if (p.win.window > 0 && p.slot_group > 1) return hipErrorInvalidValue;
  if (p.win.window > 0)
    launch_decode_kernel<ES, D, G, true, false>(p, grid, vt, lds, s);
  else if (p.slot_group > 1)
    launch_decode_kernel<ES, D, G, false, true>(p, grid, vt, lds, s);
  else
    launch_decode_kernel<ES, D, G, false, false>(p, grid, vt, lds, s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int batch = p.units / p.hkv;
  // one wave per (b, query head); the launch's threads also cover the U units
  // for the lengths copy (kThreads * blocks >= 64 * batch * hq >= units)
  const int blocks = (batch * p.hq + kWaves - 1) / kWaves;
  hipLaunchKernelGGL((combine_kernel<ES, D, G>), dim3(blocks), dim3(kThreads), 0, s, p, batch);
  return hipGetLastError();
}

template <int ES, int D>
hipError_t decode_by_group(int group, const DecodeParams &p, int grid, bool vt, hipStream_t s) {
  switch (group) {
    case 1: return decode_impl<ES, D, 1>(p, grid, vt, s);
    case 2: return decode_impl<ES, D, 2>(p, grid, vt, s);
    case 4: return decode_impl<ES, D, 4>(p, grid, vt, s);
    case 8: return decode_impl<ES, D, 8>(p, grid, vt, s);
    default: return hipErrorInvalidValue;
  }
}

template <int ES, int D>
hipError_t prefill_impl(const PrefillParams &p, bool vt, hipStream_t s) {
  // decisions and importances are staged for the passes that read them per
  // token: prompt attention (carry records enabled) and window grouping
  const bool stage = p.carry != nullptr || p.win.window > 0;
  // the neuron lines (one 128-byte line per token and unit) are kept for the
  // pages pass while they fit about twice the 256 MiB last-level cache:
  // measured, a Llama-2-7B layer (268 MB of lines) gains 50 us in the pages
  // pass from kept lines, a 70B GQA layer (1.07 GB) 28 us in this pass from
  // streamed ones
  const bool keep = int64_t(p.units) * p.n * 128 <= (int64_t(512) << 20);
  if (p.n > 0) {
    if (stage && keep)
      hipLaunchKernelGGL((prefill_decide_kernel<ES, true, kCachePolicyDefault>), dim3(p.units), dim3(kThreads), 0, s, p);
    else if (stage)
      hipLaunchKernelGGL((prefill_decide_kernel<ES, true, kNontemporal>), dim3(p.units), dim3(kThreads), 0, s, p);
    else if (keep)
      hipLaunchKernelGGL((prefill_decide_kernel<ES, false, kCachePolicyDefault>), dim3(p.units), dim3(kThreads), 0, s, p);
    else
      hipLaunchKernelGGL((prefill_decide_kernel<ES, false, kNontemporal>), dim3(p.units), dim3(kThreads), 0, s, p);
  } else {
    hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_for(p.units)), dim3(kThreads), 0, s, p.len, 0,
                       size_t(p.units));
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(alloc_pages_kernel, dim3(1), dim3(1024), 0, s, p.len, p.z, p.ptab,
                     p.page_base, p.ctrl, p.num_pages, nullptr, nullptr, 0, p.units, p.maxpages,
                     p.log2p);
  e = hipGetLastError();
  if (e != hipSuccess || p.n == 0) return e;
  // items of S_u >= l_u kItemTokens / n slots: at most ceil(n / kItemTokens)
  // per unit, and at most ceil(n / 32) (S_u >= 32, l_u <= n)
  const int items = std::min((p.n + kItemTokens - 1) / kItemTokens, (p.n + 31) / 32);
  const int64_t waves = int64_t(p.units) * items;
  const int blocks = static_cast<int>((waves + kWaves - 1) / kWaves);
  const bool win = p.win.window > 0;
  if constexpr (ES == 2) {
    if (vt && win)
      hipLaunchKernelGGL((prefill_pages_kernel<ES, D, true, true>), dim3(blocks), dim3(kThreads), 0, s,
                         p, items);
    else if (vt)
      hipLaunchKernelGGL((prefill_pages_kernel<ES, D, true, false>), dim3(blocks), dim3(kThreads), 0, s,
                         p, items);
    if (vt) return hipGetLastError();
  }
  // Row-layout caches with a window take the chunked window pass: on a
  // Llama-2-7B layer (CR 1-8, w = 12) it ran 0.32 ms against 0.36 ms for the
  // window mode of the slot-aligned pass.
  if (win) {
    const int nch = (p.n + 63) / 64;
    hipLaunchKernelGGL((prefill_window_kernel<ES, D>), dim3((nch + kWaves - 1) / kWaves, p.units),
                       dim3(kThreads), 0, s, p);
  } else {
    hipLaunchKernelGGL((prefill_pages_kernel<ES, D, false, false>), dim3(blocks), dim3(kThreads), 0, s,
                       p, items);
  }
  return hipGetLastError();
}

template <int ES, int D>
hipError_t import_impl(const DenseParams &p, bool vt, hipStream_t s) {
  const int limit = p.dense_slots < p.max_slots ? p.dense_slots : p.max_slots;
  hipLaunchKernelGGL(alloc_pages_kernel, dim3(1), dim3(1024), 0, s, p.len, p.z, p.ptab,
                     p.page_base, p.ctrl, p.num_pages, p.lengths_in, p.z_in, limit, p.units,
                     p.maxpages, p.log2p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.dense_slots == 0) return e;
  hipLaunchKernelGGL((import_kernel<ES, D>),
                     dim3((p.dense_slots + kDenseRows - 1) / kDenseRows, p.units), dim3(kThreads), 0,
                     s, p);
  e = hipGetLastError();
  if (e != hipSuccess || !vt) return e;
  return launch_transpose<D>(p.pool, p.page_bytes, p.ctrl, s);
}

template <int ES, int D>
hipError_t export_impl(const DenseParams &p, bool vt, hipStream_t s) {
  const int bx = p.dense_slots > 0 ? (p.dense_slots + kDenseRows - 1) / kDenseRows : 1;
  if (vt)
    hipLaunchKernelGGL((export_kernel<ES, D, true>), dim3(bx, p.units), dim3(kThreads), 0, s, p);
  else
    hipLaunchKernelGGL((export_kernel<ES, D, false>), dim3(bx, p.units), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace

size_t decode_lds_bytes(int table_entries, int group, int head_dim, bool window) {
  (void)group;
  // slot-space table; with a window, 2 * head_dim fp32 per wave for the
  // matrix-core decode's windowed means
  return align_up(size_t(table_entries) * 4, 16) + (window ? size_t(kWaves) * 2 * head_dim * 4 : 0);
}

size_t decode_static_lds_bytes(int head_dim, bool v_trans) {
  if (!v_trans) return 64;
  return head_dim == 128 ? mfma_ring_bytes<128>() + 64 : mfma_ring_bytes<64>() + 64;
}

hipError_t launch_fill_i32(int32_t *p, int32_t value, size_t count, hipStream_t s) {
  if (count == 0) return hipSuccess;
  hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_for(count)), dim3(kThreads), 0, s, p, value, count);
  return hipGetLastError();
}

hipError_t launch_fill_u8(void *p, size_t bytes, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  hipLaunchKernelGGL(zero_u8_kernel, dim3(grid_for(bytes)), dim3(kThreads), 0, s,
                     static_cast<uint8_t *>(p), bytes);
  return hipGetLastError();
}

hipError_t launch_copy_i32(int32_t *dst, const int32_t *src, size_t count, hipStream_t s) {
  if (count == 0) return hipSuccess;
  hipLaunchKernelGGL(copy_i32_kernel, dim3(grid_for(count)), dim3(kThreads), 0, s, dst, src, count);
  return hipGetLastError();
}

#define DMC_DISPATCH_ES_D(fn, es, d, ...)                           \
  ((es) == 2 ? ((d) == 128 ? fn<2, 128>(__VA_ARGS__) : fn<2, 64>(__VA_ARGS__)) \
             : ((d) == 128 ? fn<4, 128>(__VA_ARGS__) : fn<4, 64>(__VA_ARGS__)))

hipError_t launch_decode(int elem_bytes, int head_dim, int group, bool vt, const DecodeParams &p,
                         int grid, hipStream_t s) {
  return DMC_DISPATCH_ES_D(decode_by_group, elem_bytes, head_dim, group, p, grid, vt, s);
}

hipError_t launch_prefill(int elem_bytes, int head_dim, bool vt, const PrefillParams &p,
                          hipStream_t s) {
  return DMC_DISPATCH_ES_D(prefill_impl, elem_bytes, head_dim, p, vt, s);
}

hipError_t launch_import(int elem_bytes, int head_dim, bool vt, const DenseParams &p, hipStream_t s) {
  return DMC_DISPATCH_ES_D(import_impl, elem_bytes, head_dim, p, vt, s);
}

hipError_t launch_export(int elem_bytes, int head_dim, bool vt, const DenseParams &p, hipStream_t s) {
  return DMC_DISPATCH_ES_D(export_impl, elem_bytes, head_dim, p, vt, s);
}

}  // namespace dmc
