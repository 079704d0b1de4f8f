// gfx950 kernels of DMC prompt-phase attention.
//
// Method: Nawrot et al., "Dynamic Memory Compression" (ICML 2024).  During
// the prompt every token runs the Algorithm 1 update and then attends (the
// inference semantics of Sec. 3.1 applied at each position; Sec. 3.2 gives
// the same thing as a mask over the unrolled intermediate states, with
// discrete decisions): query i sees the final state of every segment that
// closed before it -- slots 0 .. seg(i)-1 of the compacted cache -- and the
// running (partial) mean of its own segment up to and including token i.
//
// Both kernels run after the compaction passes, which leave in the
// workspace the decisions and importance scores of every prompt token, the
// per-64-token segment-start counts, the finished cache and, for every
// 32-token boundary that falls inside a segment, the segment's running sums
// just before that boundary ("carry" records).  A query's own open state is
// therefore rebuilt from at most 31 + (tokens per wave) prompt rows, never by
// walking back to a segment start, so the cost stays linear in the prompt
// even for heads that accumulate the whole prompt into one slot.
//
// The open state enters the online softmax as its initial state (max =
// its score, sum = 1, accumulator = its value mean); the closed slots then
// stream through with a per-query limit seg(i) (a staircase mask in slot
// space).
#include <type_traits>

#include "dmc_mfma.h"

namespace dmc {
namespace {

__device__ __forceinline__ float wave_sum(float x) {
  x = row_sum<32>(x);
  return x + __shfl_xor(x, 32, 64);
}

__device__ __forceinline__ int wave_sum_int(int x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// Slot (segment index) of prompt token a + lane for lanes < cnt, -1 on the
// other lanes.  The tokens a .. a + cnt - 1 lie in one 64-token chunk.  A
// token opens a segment iff its decision is 0 (the first token always does;
// tokens past the prompt never do).
__device__ __forceinline__ int token_slots(const PromptParams &p, int u, int a, int cnt) {
  const int lane = threadIdx.x & 63;
  int before = 0;
  for (int c = lane; c < (a >> 6); c += 64) before += p.count[int64_t(u) * p.prompt_chunks + c];
  before = wave_sum_int(before);
  const int tl = (a & ~63) + lane;
  const bool st = tl < p.n && p.alpha[int64_t(u) * p.max_prompt + tl] == 0;
  const unsigned long long msk = __ballot(st);
  const int rel = a & 63;
  before += __popcll(msk & ((1ull << rel) - 1ull));
  const unsigned long long mine = msk >> rel;
  const unsigned long long upto = lane >= 63 ? ~0ull : ((2ull << lane) - 1ull);
  return lane < cnt ? before + __popcll(mine & upto) - 1 : -1;
}

// Rebuilds the open-segment running sums of tokens [a, a + cnt) (cnt >= 1)
// in token order, starting at the 32-token boundary at or below a: calls
// snap(t, ak, av, zs) for every t >= a with the sums after token t, and
// batch_end(t0) after each batch of 8 tokens t0 .. t0 + 7.  Lanes own
// elements lane * E .. lane * E + E - 1; k[0] is read as 0.
template <int ES, int D, typename Snap, typename BatchEnd>
__device__ __forceinline__ void walk_open_state(const PromptParams &p, int u, int b, int g, int a,
                                                int cnt, Snap &&snap, BatchEnd &&batch_end) {
  constexpr int E = D / 64;
  constexpr int kRows = 8;
  const int lane = threadIdx.x & 63;
  const int bs = a & ~31, end = a + cnt;
  const uint8_t *al = p.alpha + int64_t(u) * p.max_prompt;
  const float *om = p.omega + int64_t(u) * p.max_prompt;
  float ak[E], av[E], zs = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) ak[e] = av[e] = 0.0f;
  if (bs > 0 && al[bs] != 0) {   // the segment open at bs started earlier
    const float *cr = p.carry + (int64_t(u) * p.carry_blocks + (bs >> 5)) * carry_stride(D);
#pragma unroll
    for (int e = 0; e < E; ++e) {
      ak[e] = cr[lane * E + e];
      av[e] = cr[D + lane * E + e];
    }
    zs = cr[2 * D];
  }
  const char *kbase = static_cast<const char *>(p.k) + (b * p.ks[0] + g * p.ks[2] + lane * E) * ES;
  const char *vbase = static_cast<const char *>(p.v) + (b * p.vs[0] + g * p.vs[2] + lane * E) * ES;
  const int64_t kst = p.ks[1] * ES, vst = p.vs[1] * ES;
  for (int t0 = bs; t0 < end; t0 += kRows) {
    float kk[kRows][E], vv[kRows][E], ww[kRows];
    bool st[kRows];
#pragma unroll
    for (int j = 0; j < kRows; ++j) {
      const int tj = min(t0 + j, end - 1);
      load_e<ES, E>(kbase + tj * kst, kk[j]);
      load_e<ES, E>(vbase + tj * vst, vv[j]);
      ww[j] = om[tj];
      st[j] = al[tj] == 0;
    }
#pragma unroll
    for (int j = 0; j < kRows; ++j) {
      const int tj = t0 + j;
      if (tj < end) {
        if (st[j]) {
          zs = 0.0f;
#pragma unroll
          for (int e = 0; e < E; ++e) ak[e] = av[e] = 0.0f;
        }
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const float kv = (lane * E + e == 0) ? 0.0f : kk[j][e];   // k_t[0] <- 0
          ak[e] = fmaf(ww[j], kv, ak[e]);
          av[e] = fmaf(ww[j], vv[j][e], av[e]);
        }
        zs += ww[j];
        if (tj >= a) snap(tj, ak, av, zs);
      }
    }
    batch_end(t0);
  }
}

// Window grouping (Sec. 3.3): the open state of token t is the omega-
// weighted mean of its segment's tokens max(segment start, t - w + 1) .. t.
// Same interface as walk_open_state.  The walk starts at the 8-aligned token
// at or below a - w + 1 with empty sums (no carry records: a window never
// reaches further back), adds each token, restarts at segment starts and
// removes the token that leaves the window (t - w, when it lies in the
// current segment and was added), so the sums always cover the window.
template <int ES, int D, typename Snap, typename BatchEnd>
__device__ __forceinline__ void walk_window_state(const PromptParams &p, int u, int b, int g,
                                                  int a, int cnt, Snap &&snap,
                                                  BatchEnd &&batch_end) {
  constexpr int E = D / 64;
  constexpr int kRows = 8;
  const int lane = threadIdx.x & 63;
  const int W = p.window;
  const int bs = max(a - W + 1, 0) & ~7, end = a + cnt;
  const uint8_t *al = p.alpha + int64_t(u) * p.max_prompt;
  const float *om = p.omega + int64_t(u) * p.max_prompt;
  float ak[E], av[E], zs = 0.0f;
#pragma unroll
  for (int e = 0; e < E; ++e) ak[e] = av[e] = 0.0f;
  int first = bs;   // first token in the sums: the walk's start or the segment's
  const char *kbase = static_cast<const char *>(p.k) + (b * p.ks[0] + g * p.ks[2] + lane * E) * ES;
  const char *vbase = static_cast<const char *>(p.v) + (b * p.vs[0] + g * p.vs[2] + lane * E) * ES;
  const int64_t kst = p.ks[1] * ES, vst = p.vs[1] * ES;
  for (int t0 = bs; t0 < end; t0 += kRows) {
    float kk[kRows][E], vv[kRows][E], ww[kRows];
    float ko[kRows][E], vo[kRows][E], wo[kRows];
    bool st[kRows];
#pragma unroll
    for (int j = 0; j < kRows; ++j) {
      const int tj = min(t0 + j, end - 1);
      const int to = max(tj - W, 0);
      load_e<ES, E>(kbase + tj * kst, kk[j]);
      load_e<ES, E>(vbase + tj * vst, vv[j]);
      load_e<ES, E>(kbase + to * kst, ko[j]);
      load_e<ES, E>(vbase + to * vst, vo[j]);
      ww[j] = om[tj];
      wo[j] = om[to];
      st[j] = al[tj] == 0;
    }
#pragma unroll
    for (int j = 0; j < kRows; ++j) {
      const int tj = t0 + j;
      if (tj < end) {
        if (st[j]) {
          zs = 0.0f;
#pragma unroll
          for (int e = 0; e < E; ++e) ak[e] = av[e] = 0.0f;
          first = tj;
        }
        if (lane == 0) {   // k_t[0] <- 0
          kk[j][0] = 0.0f;
          ko[j][0] = 0.0f;
        }
#pragma unroll
        for (int e = 0; e < E; ++e) {
          ak[e] = fmaf(ww[j], kk[j][e], ak[e]);
          av[e] = fmaf(ww[j], vv[j][e], av[e]);
        }
        zs += ww[j];
        if (tj - W >= first) {   // token tj - W leaves the window
#pragma unroll
          for (int e = 0; e < E; ++e) {
            ak[e] = fmaf(-wo[j], ko[j][e], ak[e]);
            av[e] = fmaf(-wo[j], vo[j][e], av[e]);
          }
          zs -= wo[j];
        }
        if (tj >= a) snap(tj, ak, av, zs);
      }
    }
    batch_end(t0);
  }
}

// ---------------------------------------------------------------------------
// bf16 on matrix cores.  One workgroup = 4 waves = one unit's 128 query
// columns (token-major: column c is token c / G, head c % G of the group);
// each wave owns 32 columns, T = 32 / G tokens.  The unit's closed slots
// stream through LDS in blocks of 32, shared by the 4 waves; per block and
// wave, on v_mfma_f32_32x32x16_bf16 (lane l: column l % 32, half l / 32),
//   S^T[slot][col]  = K[slot][:] . Q[col][:]          (A = K, B = Q^T)
//   O^T[dim][col]  += V^T[dim][slot] P^T[slot][col]    (A = V^T, B = P^T)
// Score row m of a block is key slot pi(m) (bits 2 and 3 of m swapped):
// then a lane's score registers 8 kk .. 8 kk + 7 are exactly its P^T
// operand for value k-step kk (slots 16 kk + 8 half .. + 8).
//
// Blocks arrive by direct global -> LDS transfers (16 bytes per lane, no
// registers) into a ring of kStages buffers, kStages - 1 blocks ahead of the
// one being multiplied.  Rows land XOR-swizzled in 16-byte units so that the
// operand loads of each 16-lane group hit distinct banks.  Value rows are
// read transposed by ds_read_b64_tr_b16 (a 16-lane group pointing at four
// 8-byte row pieces of each of 4 rows receives, per lane, one column's 4
// consecutive rows); caches that store value pages transposed ([d][P]) are
// read as V^T rows directly.  The softmax rescales the accumulators only
// when some column's running maximum grows by more than 2^8 (probabilities
// stay below 256, exact enough in bf16 and fp32).  Workgroups are mapped so
// that all tiles of a unit run on one XCD (sharing its L2), latest tiles
// (most slots) first.  P enters the value product rounded to bf16 and its
// sum is taken over the rounded values.
// ---------------------------------------------------------------------------
#ifndef DMC_PROMPT_STAGES
#define DMC_PROMPT_STAGES 4
#endif
constexpr int kStages = DMC_PROMPT_STAGES;
constexpr int kPtabLds = kPromptMaxPages;   // page-table entries of a unit cached in LDS

// Open states of a wave's columns on the matrix cores (exact Algorithm 1).
// The wave's tokens lie in one 32-token block starting at bs = a & ~31, and
// the open state of token t is the omega-weighted mean of its segment's
// tokens up to t: those of the block from the segment start (or from bs,
// plus the carry record at bs, when the segment began earlier).  With
// W[t][j] = omega_{bs+j} over that range of block rows j and 0 elsewhere:
//   score(t) = (sum_j W[t][j] (q_t . k_{bs+j}) + q_t . carry_k) / z_t
//   value(t) = (sum_j W[t][j] v_{bs+j} + carry_v) / z_t
//   z_t      =  sum_j W[t][j] + carry_z
// q_t . k_j comes from the same score product as the closed slots (raw key
// rows as A operands, straight from global memory; q[0] is already zeroed,
// which leaves k[0] out).  The value sum is V^T[dim][j] W^T[j][col] on the
// matrix cores with W split into a bf16 head and tail (W = hi + lo to about
// 2^-17), the raw value rows staged in LDS (value swizzle) for transposed
// reads.  Results go into the online softmax state as in the vector walk:
// max = score, weight 1 (counted in one half), accumulator = value mean.
template <int D, int G>
__device__ __forceinline__ void open_state_mfma(const PromptParams &p, int u, int b, int g, int a,
                                                int nb, int col, int hb, int tok,
                                                bool colv, const uint4 (&qop)[D / 16],
                                                char *vstage, float &m, float &ls,
                                                f32x16_t (&acc)[D / 32]) {
  constexpr int KS = D / 16, NTL = D / 32, RB = D * 2, CPR = D / 8;
  constexpr int NDMA = 32 * RB / 1024;   // 16-byte transfers per lane for 32 value rows
  const int lane = threadIdx.x & 63;
  const int bs = a & ~31;
  const int last = nb - 1;               // rows past the prompt read its last row (weight 0)
  const uint8_t *al = p.alpha + int64_t(u) * p.max_prompt;
  const float *om = p.omega + int64_t(u) * p.max_prompt;
  const char *kbase = static_cast<const char *>(p.k) + (b * p.ks[0] + g * p.ks[2]) * 2;
  const char *vbase = static_cast<const char *>(p.v) + (b * p.vs[0] + g * p.vs[2]) * 2;
  const int64_t kst = p.ks[1] * 2, vst = p.vs[1] * 2;

  // Raw value rows bs .. bs + 31 into this wave's staging block.
#pragma unroll
  for (int i = 0; i < NDMA; ++i) {
    const int c = i * 64 + lane;
    const int row = c / CPR, pc = c - row * CPR;
    const int trow = min(bs + row, last);
    dma16(vstage + i * 1024, vbase + trow * vst + (pc ^ v_swizzle<CPR>(row)) * 16);
  }
  // Raw key row bs + pi(col) as this lane's A operand.
  uint4 kop[KS];
  {
    const char *kr = kbase + min(bs + score_slot(col), last) * kst + hb * 16;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kop[ks] = ld16(kr + ks * 32);
  }
  // Segment starts of the block (bit j: token bs + j opens a segment).
  const int ta = min(bs + (lane & 31), last);
  const uint32_t starts = static_cast<uint32_t>(__ballot(lane < 32 && bs + lane <= last && al[ta] == 0));
  // This column's token and the first block row of its open segment.
  const int tr = colv ? a + tok - bs : -1;
  const uint32_t upto = tr >= 0 ? starts & (0xffffffffu >> (31 - tr)) : 0u;
  const int first = upto ? 31 - __clz(upto) : 0;
  const bool carried = colv && upto == 0 && bs > 0;
  // Weights of the lane's rows j = 16 kk + 8 hb + e (register 8 kk + e of the
  // score product holds row j, as in the closed-slot blocks).
  float w[16];
  float zs = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int j = 16 * (i >> 3) + 8 * hb + (i & 7);
    const float wj = om[min(bs + j, last)];
    w[i] = (j >= first && j <= tr) ? wj : 0.0f;
    zs += w[i];
  }

  f32x16_t sc = f32x16_t{};
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) sc = mfma_32x32x16(kop[ks], qop[ks], sc);
  float part = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) part = fmaf(w[i], sc[i], part);

  // W^T operands, head and tail.
  uint4 whi[2], wlo[2];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    uint32_t h[4], l[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float w0 = w[8 * kk + 2 * q], w1 = w[8 * kk + 2 * q + 1];
      h[q] = cvt_pk_bf16(w0, w1);
      const float h0 = __uint_as_float(h[q] << 16), h1 = __uint_as_float(h[q] & 0xffff0000u);
      l[q] = cvt_pk_bf16(w0 - h0, w1 - h1);
    }
    whi[kk] = make_uint4(h[0], h[1], h[2], h[3]);
    wlo[kk] = make_uint4(l[0], l[1], l[2], l[3]);
  }

  // Carry record of the block when some column's segment began before bs.
  float cz = 0.0f;
  f32x16_t cv[NTL];
#pragma unroll
  for (int t = 0; t < NTL; ++t) cv[t] = f32x16_t{};
  if (__any(carried)) {
    const float *cr = p.carry + (int64_t(u) * p.carry_blocks + (bs >> 5)) * carry_stride(D);
    if (carried) {
      float qk = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        float qf[8];
        V16<2>::unpack(qop[ks], qf);
        const float4 k0 = *reinterpret_cast<const float4 *>(cr + 16 * ks + 8 * hb);
        const float4 k1 = *reinterpret_cast<const float4 *>(cr + 16 * ks + 8 * hb + 4);
        qk = fmaf(qf[0], k0.x, qk);
        qk = fmaf(qf[1], k0.y, qk);
        qk = fmaf(qf[2], k0.z, qk);
        qk = fmaf(qf[3], k0.w, qk);
        qk = fmaf(qf[4], k1.x, qk);
        qk = fmaf(qf[5], k1.y, qk);
        qk = fmaf(qf[6], k1.z, qk);
        qk = fmaf(qf[7], k1.w, qk);
      }
      part += qk;
#pragma unroll
      for (int t = 0; t < NTL; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float4 x = *reinterpret_cast<const float4 *>(cr + D + 32 * t + 8 * i + 4 * hb);
          cv[t][4 * i + 0] = x.x;
          cv[t][4 * i + 1] = x.y;
          cv[t][4 * i + 2] = x.z;
          cv[t][4 * i + 3] = x.w;
        }
      cz = cr[2 * D];
    }
  }
  part += __shfl_xor(part, 32, 64);
  zs += __shfl_xor(zs, 32, 64) + cz;

  // Value sums: A = V^T[dim 32 t + col][rows 16 kk + 8 hb .. + 8] (transposed reads).
  wait_vmcnt<0>();
  wave_lds_sync();
  uint32_t vaddr[NTL];
  {
    const int g16 = lane >> 4, r16 = lane & 15;
    const int row0 = 8 * (g16 >> 1) + (r16 >> 2);
#pragma unroll
    for (int t = 0; t < NTL; ++t) {
      const int lc = 4 * t + 2 * (g16 & 1) + ((r16 & 3) >> 1);
      vaddr[t] = row0 * RB + ((lc ^ v_swizzle<CPR>(row0)) * 16) + (r16 & 1) * 8;
    }
  }
#pragma unroll
  for (int t = 0; t < NTL; ++t) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const uint2 h0 = ds_read_tr16(vstage + vaddr[t] + 16 * kk * RB);
      const uint2 h1 = ds_read_tr16(vstage + vaddr[t] + (16 * kk + 4) * RB);
      const uint4 va = make_uint4(h0.x, h0.y, h1.x, h1.y);
      cv[t] = mfma_32x32x16(va, whi[kk], cv[t]);
      cv[t] = mfma_32x32x16(va, wlo[kk], cv[t]);
    }
  }
  if (colv) {
    const float inv = 1.0f / zs;
    m = part * inv * p.scale_log2;
    ls = hb == 0 ? 1.0f : 0.0f;   // the open state's weight, counted once per column
#pragma unroll
    for (int t = 0; t < NTL; ++t) acc[t] = cv[t] * inv;
  }
}

// BIG: pages of >= 32 slots (one page per 32-slot block); VT: value pages
// stored transposed (32-slot pages only).
template <int D, int G, bool VT, bool BIG>
__global__ __launch_bounds__(kThreads, 2) void prompt_mfma_kernel(PromptParams p, int ntiles) {
  static_assert(!VT || BIG, "transposed value pages hold 32 slots");
  constexpr int T = 32 / G;            // tokens per wave
  constexpr int TW = kWaves * T;       // tokens per workgroup
  constexpr int KS = D / 16;           // 16-dim k-steps of the score product
  constexpr int NTL = D / 32;          // 32-dim tiles of the value product
  constexpr int RB = D * 2;
  constexpr int CPR = D / 8;           // 16-byte chunks per row
  constexpr int BLK = 32 * RB;         // bytes of one block's keys (and of its values)
  constexpr int DPW = BLK / 16 / kThreads;   // transfers per thread per block half
  constexpr int SLOT = 2 * BLK;         // one ring slot: a block's keys, then its values
  constexpr int STAGE = 8 * 2 * D;     // floats per wave: 8 tokens x (key mean, value mean)
  static_assert(STAGE * 4 == BLK && kWaves == 4, "open-state staging: two waves per ring slot");
  static_assert(DPW >= 1 && BLK % (16 * kThreads) == 0, "block split");
  static_assert(kStages == 3 || kStages == 4, "ring depth");
  // The block ring, one array per slot (see dma16_s).
  __shared__ __align__(16) unsigned char ring0[SLOT], ring1[SLOT], ring2[SLOT];
  __shared__ __align__(16) unsigned char ring3[kStages > 3 ? SLOT : 16];
  auto slot = [&](auto st_c) -> unsigned char * {
    constexpr int S = decltype(st_c)::value;
    if constexpr (S == 0) return ring0;
    else if constexpr (S == 1) return ring1;
    else if constexpr (S == 2) return ring2;
    else return ring3;
  };
  __shared__ int s_hi[kWaves];
  __shared__ int s_pt[kPtabLds];

  const int bid = blockIdx.x;
  const int xcd = bid & 7, r = bid >> 3;
  const int ul = r / ntiles, tile = ntiles - 1 - (r - ul * ntiles);
  const int u = ul * 8 + xcd;
  if (u >= p.units) return;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, hb = lane >> 5;   // MFMA column and half
  const int b = u / p.hkv, g = u - b * p.hkv;
  const int nb = clamp_prompt_len(p.prompt_lens, p.n, b);
  const bool ok = p.page_base[u] >= 0;
  const int a = tile * TW + wave * T;
  const int cnt = ok ? max(0, min(T, nb - a)) : 0;
  const uint4 zero4 = make_uint4(0, 0, 0, 0);
  // This wave's staging area for the open states (before the ring runs).
  unsigned char *wstage = (wave < 2 ? ring0 : ring1) + (wave & 1) * BLK;

  // The tile's page-table slice, loaded now for a bound on the slots it can
  // see (a token's slot never exceeds the token) and stored to LDS before the
  // first barrier.
  const int P = 1 << p.log2p;
  const int64_t pt = int64_t(u) * p.maxpages;
  const int npg = min(min((min(nb, tile * TW + TW) + P - 1) >> p.log2p, p.maxpages), kPtabLds);
  constexpr int kPtPer = (kPtabLds + kThreads - 1) / kThreads;
  int ptv[kPtPer];
#pragma unroll
  for (int j = 0; j < kPtPer; ++j) {
    const int i = tid + j * kThreads;
    ptv[j] = i < npg ? p.ptab[pt + i] : 0;
  }

  const int seg = cnt > 0 ? token_slots(p, u, a, cnt) : -1;
  const int tok = col / G, head = col - tok * G;
  const bool colv = tok < cnt;
  const int lim = colv ? __shfl(seg, tok, 64) : 0;
  const int wave_hi = __builtin_amdgcn_readfirstlane(cnt > 0 ? __shfl(seg, cnt - 1, 64) : 0);
  // every column of the wave sees slots < wave_lo (0 when some column is empty)
  const int wave_lo = __builtin_amdgcn_readfirstlane(cnt == T ? __shfl(seg, 0, 64) : 0);
  if (lane == 0) s_hi[wave] = wave_hi;

  // Q^T operand: lane holds Q[col][16 ks + 8 hb .. + 8] (q[0] is not part of the score).
  uint4 qop[KS];
  {
    const char *qr = static_cast<const char *>(p.q) +
                     (b * p.qs[0] + int64_t(a + tok) * p.qs[1] + (g * G + head) * p.qs[2]) * 2;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qop[ks] = colv ? ld16(qr + ks * 32 + hb * 16) : zero4;
    if (hb == 0) qop[0].x &= 0xffff0000u;
  }

  float m = 0.0f, ls = 0.0f;
  f32x16_t acc[NTL];
#pragma unroll
  for (int t = 0; t < NTL; ++t) acc[t] = f32x16_t{};

  // Open state of each column's token.
  if (cnt > 0 && p.window == 0) {
    open_state_mfma<D, G>(p, u, b, g, a, nb, col, hb, tok, colv, qop,
                          reinterpret_cast<char *>(wstage), m, ls, acc);
  } else if (cnt > 0) {
    // Window grouping: the walk stages key and value means of 8 tokens at a
    // time (fp32, this wave's part of the block ring); then every lane takes
    // its column's score (dot with its Q^T slice, summed over the two halves)
    // and its slice of the value mean.
    float *stage = reinterpret_cast<float *>(wstage);
    constexpr int E = D / 64;
    auto snap = [&](int t, const float *ak, const float *av, float zs) {
          const float inv = 1.0f / zs;
          float *row = stage + (t & 7) * 2 * D;
#pragma unroll
          for (int e = 0; e < E; ++e) {
            row[lane * E + e] = ak[e] * inv;
            row[D + lane * E + e] = av[e] * inv;
          }
        };
    auto batch_end = [&](int t0) {
          if (t0 + 8 <= a) return;   // nothing staged in this batch
          wave_lds_sync();
          const int t = a + tok;
          const bool here = colv && t >= t0 && t < t0 + 8;
          float part = 0.0f;
          if (here) {
            const float *kp = stage + (t & 7) * 2 * D;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
              float qf[8];
              V16<2>::unpack(qop[ks], qf);
              const float4 k0 = *reinterpret_cast<const float4 *>(kp + 16 * ks + 8 * hb);
              const float4 k1 = *reinterpret_cast<const float4 *>(kp + 16 * ks + 8 * hb + 4);
              part = fmaf(qf[0], k0.x, part);
              part = fmaf(qf[1], k0.y, part);
              part = fmaf(qf[2], k0.z, part);
              part = fmaf(qf[3], k0.w, part);
              part = fmaf(qf[4], k1.x, part);
              part = fmaf(qf[5], k1.y, part);
              part = fmaf(qf[6], k1.z, part);
              part = fmaf(qf[7], k1.w, part);
            }
          }
          part += __shfl_xor(part, 32, 64);
          if (here) {
            const float *vp = stage + (t & 7) * 2 * D + D;
            m = part * p.scale_log2;
            ls = hb == 0 ? 1.0f : 0.0f;   // the open state's weight, counted once per column
#pragma unroll
            for (int tt = 0; tt < NTL; ++tt)
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const float4 x = *reinterpret_cast<const float4 *>(vp + 32 * tt + 8 * i + 4 * hb);
                acc[tt][4 * i + 0] = x.x;
                acc[tt][4 * i + 1] = x.y;
                acc[tt][4 * i + 2] = x.z;
                acc[tt][4 * i + 3] = x.w;
              }
          }
          wave_lds_sync();
        };
    walk_window_state<2, D>(p, u, b, g, a, cnt, snap, batch_end);
  }
#pragma unroll
  for (int j = 0; j < kPtPer; ++j) {
    const int i = tid + j * kThreads;
    if (i < npg) s_pt[i] = ptv[j];
  }
  __syncthreads();   // slot limits and page table published; staging area free again

  int s_top = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) s_top = max(s_top, s_hi[w]);
  s_top = __builtin_amdgcn_readfirstlane(s_top);
  const int nblk = (s_top + 31) >> 5;

  // Transfers of block kb into ring slot st.  This thread's chunks and their
  // byte offsets within a 32-row block (rows XOR-swizzled; LDS position =
  // chunk index).  Pages of >= 32 slots hold a block in one page: one
  // wave-uniform base plus fixed per-lane offsets.  Smaller pages: one base
  // per transfer (below).  Rows past the closed slots are masked or zeroed
  // when used.
  uint32_t koff[DPW], voff[DPW];
  int krow_of[DPW];
#pragma unroll
  for (int i = 0; i < DPW; ++i) {
    const int c = (i * kWaves + wave) * 64 + lane;
    const int row = c / CPR, pc = c - row * CPR;
    krow_of[i] = row;
    koff[i] = row * RB + (pc ^ k_swizzle<CPR>(row)) * 16;
    if (VT) {
      const int dim = c >> 2, lc = (c & 3) ^ vt_swizzle(dim);
      voff[i] = dim * 64 + lc * 16;   // value page [D][32]
    } else {
      voff[i] = row * RB + (pc ^ v_swizzle<CPR>(row)) * 16;
    }
  }
  // Every call issues the same 2 DPW transfers per wave; those of blocks
  // past the last one are switched off (no memory read).  Pages of fewer
  // than 32 slots: one transfer covers 1024 / RB <= 8 consecutive rows,
  // which lie in one page (pages hold >= 8 slots), so its base is that
  // page; rows past the closed slots are switched off per lane.
  auto issue = [&](int kb, auto st_c) {
    unsigned char *dst = slot(st_c);
    const bool on = kb < nblk;
    if constexpr (BIG) {
      const int s0 = kb * 32;
      const int pg = on ? __builtin_amdgcn_readfirstlane(s_pt[min(s0 >> p.log2p, kPtabLds - 1)]) : 0;
      const char *page = p.pool + int64_t(pg) * p.page_bytes;
      const char *kb_base = uniform_ptr(page + int64_t(s0 & (P - 1)) * RB);
      const char *vb_base = uniform_ptr(VT ? page + int64_t(P) * RB : kb_base + int64_t(P) * RB);
#pragma unroll
      for (int i = 0; i < DPW; ++i) {
        unsigned char *kdst = dst + (i * kWaves + wave) * 1024;
        dma16_s(kdst, kb_base, koff[i], on);
        dma16_s(kdst + BLK, vb_base, voff[i], on);
      }
    } else {
#pragma unroll
      for (int i = 0; i < DPW; ++i) {
        unsigned char *kdst = dst + (i * kWaves + wave) * 1024;
        const int r0 = (i * kWaves + wave) * (1024 / RB);   // first row of the transfer
        const int s = kb * 32 + r0;
        const bool live = on && s < s_top;
        const int pg = live ? __builtin_amdgcn_readfirstlane(s_pt[s >> p.log2p]) : 0;
        const char *base = uniform_ptr(p.pool + int64_t(pg) * p.page_bytes +
                                       int64_t(live ? s & (P - 1) : 0) * RB);
        const bool lane_on = kb * 32 + krow_of[i] < s_top;
        const uint32_t rel = uint32_t(r0 * RB);
        dma16_s(kdst, base, lane_on ? koff[i] - rel : kOutOfRange, live);
        dma16_s(kdst + BLK, base, lane_on ? uint32_t(P * RB) + voff[i] - rel : kOutOfRange, live);
      }
    }
  };

  // Loop-invariant LDS read offsets (within a ring slot).  Keys: row
  // pi(col), chunk (2 ks + hb) ^ swizzle -> 8 offsets.  Values (rows, read
  // transposed): row 16 kk + 8 hb + 4 hf + (lane & 15) / 4 has swizzle
  // 4 * ((lane >> 2) & 3) independent of kk and hf, so the 16 reads need one
  // offset per tile t (kk, hf as immediates).  V^T rows: one offset per kk.
  const int krow = score_slot(col);
  uint32_t kaddr[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) kaddr[ks] = krow * RB + (((2 * ks + hb) ^ k_swizzle<CPR>(krow)) * 16);
  uint32_t vaddr[VT ? 2 : NTL];
  if (VT) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) vaddr[kk] = col * 64 + (((2 * kk + hb) ^ vt_swizzle(col)) * 16);
  } else {
    const int g16 = lane >> 4, r16 = lane & 15;
    const int row0 = 8 * (g16 >> 1) + (r16 >> 2);
#pragma unroll
    for (int t = 0; t < NTL; ++t) {
      const int lc = 4 * t + 2 * (g16 & 1) + ((r16 & 3) >> 1);
      vaddr[t] = row0 * RB + ((lc ^ v_swizzle<CPR>(row0)) * 16) + (r16 & 1) * 8;
    }
  }

  const float sl2 = p.scale_log2;
  auto scores = [&](const char *kd) {
    f32x16_t sc = f32x16_t{};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      sc = mfma_32x32x16(*reinterpret_cast<const uint4 *>(kd + kaddr[ks]), qop[ks], sc);
    return sc;
  };

  // Pipelined over blocks: step kb runs block kb's exponentials between the
  // score MFMAs of block kb + 1 (one accumulator chain, order pinned by
  // scheduling barriers, key operands read two ahead), then block kb's value
  // product.
  // kStages - 1 blocks are always in flight ahead of the one multiplied
  // (2 DPW transfers each), so the waits are fixed counts.
  issue(0, std::integral_constant<int, 0>{});
  issue(1, std::integral_constant<int, 1>{});
  if constexpr (kStages > 3) issue(2, std::integral_constant<int, 2>{});
  f32x16_t scn = f32x16_t{};
  if (nblk > 0) {
    wait_vmcnt<(kStages - 2) * 2 * DPW>();
    ring_barrier();   // block 0 is in LDS for every wave
    if (wave_hi > 0) scn = scores(reinterpret_cast<const char *>(ring0));
  }
  auto step = [&](auto stage_c, int kb) {
    constexpr int ST = decltype(stage_c)::value, SN = (ST + 1) % kStages;
    wait_vmcnt<(kStages - 3) * 2 * DPW>();   // block kb + 1 has landed
    ring_barrier();   // every wave is past step kb - 1: the ring slot of kb - 1 is free
    issue(kb + kStages - 1, std::integral_constant<int, (ST + kStages - 1) % kStages>{});
    if (kb * 32 >= wave_hi) return;
    const char *vd = reinterpret_cast<const char *>(slot(stage_c)) + BLK;
    const char *kn = reinterpret_cast<const char *>(slot(std::integral_constant<int, SN>{}));   // block kb + 1's keys

    // Raw scores; slots past this column's limit are masked only in blocks
    // that reach the staircase.
    float sv[16];
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) sv[rr] = scn[rr];
    if (kb * 32 + 32 > wave_lo) {   // the block reaches the staircase
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const int slot = kb * 32 + score_slot(8 * (rr >> 2) + 4 * hb + (rr & 3));
        if (slot >= lim) sv[rr] = neg_inf();
      }
    }
    float mx = fmaxf(fmaxf(sv[0], sv[1]), sv[2]);
#pragma unroll
    for (int rr = 3; rr < 15; rr += 2) mx = fmaxf(fmaxf(mx, sv[rr]), sv[rr + 1]);
    mx = fmaxf(mx, sv[15]);
    mx = max_halves(mx) * sl2;
    if (__any(mx > m + kLazyRescale)) {
      const float mn = fmaxf(m, mx);
      const float f = fast_exp2(m - mn);
      m = mn;
      ls *= f;
#pragma unroll
      for (int t = 0; t < NTL; ++t) acc[t] *= f;
    }
    // The next block's slot always holds readable data; past the last block
    // its scores are not used.
    uint4 kr[3];
    kr[0] = *reinterpret_cast<const uint4 *>(kn + kaddr[0]);
    kr[1] = *reinterpret_cast<const uint4 *>(kn + kaddr[1]);
    f32x16_t sc = f32x16_t{};
    float ev[16];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ks + 2 < KS) kr[(ks + 2) % 3] = *reinterpret_cast<const uint4 *>(kn + kaddr[ks + 2]);
      sc = mfma_32x32x16(kr[ks % 3], qop[ks], sc);
#pragma unroll
      for (int e = 0; e < 16 / KS; ++e) {
        const int i = ks * (16 / KS) + e;
        ev[i] = fast_exp2(fmaf(sv[i], sl2, -m));
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    scn = sc;
    uint4 pb[2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      uint32_t w[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        w[q] = cvt_pk_bf16(ev[8 * kk + 2 * q], ev[8 * kk + 2 * q + 1]);
        ls = add_pair(w[q], ls);
      }
      pb[kk] = make_uint4(w[0], w[1], w[2], w[3]);
    }

    // Value product: A = V^T[dim 32 t + col][slots 16 kk + 8 hb .. + 8].
    uint4 va[NTL][2];
#pragma unroll
    for (int t = 0; t < NTL; ++t) {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        if (VT) {
          va[t][kk] = *reinterpret_cast<const uint4 *>(vd + 2048 * t + vaddr[kk]);
        } else {
          const uint2 h0 = ds_read_tr16(vd + vaddr[t] + 16 * kk * RB);
          const uint2 h1 = ds_read_tr16(vd + vaddr[t] + (16 * kk + 4) * RB);
          va[t][kk] = make_uint4(h0.x, h0.y, h1.x, h1.y);
        }
      }
    }
    if (kb * 32 + 32 > s_top) {   // the last block: clear the slots past the closed ones
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const int keep = s_top - (kb * 32 + 16 * kk + 8 * hb);
        uint32_t msk[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          msk[q] = (2 * q < keep ? 0x0000ffffu : 0u) | (2 * q + 1 < keep ? 0xffff0000u : 0u);
#pragma unroll
        for (int t = 0; t < NTL; ++t) {
          va[t][kk].x &= msk[0];
          va[t][kk].y &= msk[1];
          va[t][kk].z &= msk[2];
          va[t][kk].w &= msk[3];
        }
      }
    }
#pragma unroll
    for (int t = 0; t < NTL; ++t)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) acc[t] = mfma_32x32x16(va[t][kk], pb[kk], acc[t]);
  };

  // Whole rounds of kStages steps (a step past the last block only keeps the
  // barriers and transfer counts in step), so that no transfer is issued on
  // one path and not on another.
  for (int kb = 0; kb < nblk; kb += kStages) {
    step(std::integral_constant<int, 0>{}, kb);
    step(std::integral_constant<int, 1>{}, kb + 1);
    step(std::integral_constant<int, 2>{}, kb + 2);
    if constexpr (kStages > 3) step(std::integral_constant<int, 3>{}, kb + 3);
  }

  // Normalise and store: lane holds dims 32 t + 8 i + 4 hb .. + 4 of its column.
  float lt = ls + __shfl_xor(ls, 32, 64);
  const int t = a + tok;
  if (t < p.n) {
    const float inv = colv ? 1.0f / lt : 0.0f;
    char *orow = static_cast<char *>(p.out) +
                 (b * p.os[0] + int64_t(t) * p.os[1] + (g * G + head) * p.os[2]) * 2;
#pragma unroll
    for (int tt = 0; tt < NTL; ++tt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t lo = cvt_pk_bf16(acc[tt][4 * i] * inv, acc[tt][4 * i + 1] * inv);
        const uint32_t hi = cvt_pk_bf16(acc[tt][4 * i + 2] * inv, acc[tt][4 * i + 3] * inv);
        *reinterpret_cast<uint2 *>(orow + (32 * tt + 8 * i + 4 * hb) * 2) = make_uint2(lo, hi);
      }
  }
}

// ---------------------------------------------------------------------------
// Vector-ALU kernel (every dtype; used for fp32).  One wave = one unit's
// TG = max(1, 8 / G) tokens with all G heads of the group (R = TG * G <= 8
// query rows); lanes own head-dim elements; closed slots stream row by row
// with R online-softmax states.
// ---------------------------------------------------------------------------
template <int ES, int D, int G>
__global__ __launch_bounds__(kThreads) void prompt_valu_kernel(PromptParams p, int ngroups) {
  constexpr int TG = G >= 8 ? 1 : 8 / G;
  constexpr int R = TG * G;
  constexpr int E = D / 64;
  constexpr int RB = D * ES;
  constexpr int kAhead = 4;   // slot rows in flight
  const int lane = threadIdx.x & 63;
  const int wid = blockIdx.x * kWaves + (threadIdx.x >> 6);
  const int u = wid / ngroups;
  if (u >= p.units) return;
  const int grp = wid - u * ngroups;
  const int b = u / p.hkv, g = u - b * p.hkv;
  const int nb = clamp_prompt_len(p.prompt_lens, p.n, b);
  const bool ok = p.page_base[u] >= 0;
  const int a = grp * TG;
  const int cnt = ok ? max(0, min(TG, nb - a)) : 0;

  float qr[R][E];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j = r / G, h = r - j * G;
#pragma unroll
    for (int e = 0; e < E; ++e) qr[r][e] = 0.0f;
    if (j < cnt)
      load_e<ES, E>(static_cast<const char *>(p.q) +
                        (b * p.qs[0] + int64_t(a + j) * p.qs[1] + (g * G + h) * p.qs[2] + lane * E) * ES,
                    qr[r]);
    if (lane == 0) qr[r][0] = 0.0f;   // q[0] is not part of the score
  }

  float m[R], l[R], acc[R][E];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    m[r] = 0.0f;
    l[r] = 1.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[r][e] = 0.0f;
  }
  int seg = -1, lim[TG];
  if (cnt > 0) {
    seg = token_slots(p, u, a, cnt);
    auto snap = [&](int t, const float *ak, const float *av, float zs) {
          const float inv = 1.0f / zs;
#pragma unroll
          for (int r = 0; r < R; ++r) {
            if (a + r / G != t) continue;
            float d = 0.0f;
#pragma unroll
            for (int e = 0; e < E; ++e) d = fmaf(qr[r][e], ak[e] * inv, d);
            m[r] = wave_sum(d) * p.scale_log2;
#pragma unroll
            for (int e = 0; e < E; ++e) acc[r][e] = av[e] * inv;
          }
        };
    if (p.window > 0)
      walk_window_state<ES, D>(p, u, b, g, a, cnt, snap, [](int) {});
    else
      walk_open_state<ES, D>(p, u, b, g, a, cnt, snap, [](int) {});
  }
  int hi = 0;
#pragma unroll
  for (int j = 0; j < TG; ++j) {
    const int sj = __shfl(seg, j, 64);
    lim[j] = j < cnt ? sj : 0;
    hi = max(hi, lim[j]);
  }
  const int P = 1 << p.log2p;
  const int64_t pt = int64_t(u) * p.maxpages;
  for (int s0 = 0; s0 < hi; s0 += kAhead) {
    float kk[kAhead][E], vv[kAhead][E];
#pragma unroll
    for (int i = 0; i < kAhead; ++i) {
      const int s = min(s0 + i, hi - 1);
      const char *row = p.pool + int64_t(p.ptab[pt + (s >> p.log2p)]) * p.page_bytes +
                        int64_t(s & (P - 1)) * RB + lane * E * ES;
      load_e<ES, E>(row, kk[i]);
      load_e<ES, E>(row + int64_t(P) * RB, vv[i]);
    }
#pragma unroll
    for (int i = 0; i < kAhead; ++i) {
      const int s = s0 + i;
      if (s >= hi) break;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (s >= lim[r / G]) continue;
        float d = 0.0f;
#pragma unroll
        for (int e = 0; e < E; ++e) d = fmaf(qr[r][e], kk[i][e], d);
        const float x = wave_sum(d) * p.scale_log2;
        const float mn = fmaxf(m[r], x);
        const float f = fast_exp2(m[r] - mn), w = fast_exp2(x - mn);
        l[r] = l[r] * f + w;
#pragma unroll
        for (int e = 0; e < E; ++e) acc[r][e] = fmaf(acc[r][e], f, w * vv[i][e]);
        m[r] = mn;
      }
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j = r / G, h = r - j * G;
    const int t = a + j;
    if (t >= p.n) continue;
    float o[E];
    const float inv = j < cnt ? 1.0f / l[r] : 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) o[e] = acc[r][e] * inv;
    store_e<ES, E>(static_cast<char *>(p.out) +
                       (b * p.os[0] + int64_t(t) * p.os[1] + (g * G + h) * p.os[2] + lane * E) * ES,
                   o);
  }
}

template <int D, int G>
hipError_t prompt_mfma(const PromptParams &p, bool vt, hipStream_t s) {
  constexpr int TW = kWaves * (32 / G);
  const int ntiles = (p.n + TW - 1) / TW;
  const int64_t blocks = int64_t(8) * ((p.units + 7) / 8) * ntiles;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  if (vt)
    hipLaunchKernelGGL((prompt_mfma_kernel<D, G, true, true>), dim3(unsigned(blocks)),
                       dim3(kThreads), 0, s, p, ntiles);
  else if (p.log2p >= 5)
    hipLaunchKernelGGL((prompt_mfma_kernel<D, G, false, true>), dim3(unsigned(blocks)),
                       dim3(kThreads), 0, s, p, ntiles);
  else
    hipLaunchKernelGGL((prompt_mfma_kernel<D, G, false, false>), dim3(unsigned(blocks)),
                       dim3(kThreads), 0, s, p, ntiles);
  return hipGetLastError();
}

template <int ES, int D, int G>
hipError_t prompt_valu(const PromptParams &p, hipStream_t s) {
  constexpr int TG = G >= 8 ? 1 : 8 / G;
  const int ngroups = (p.n + TG - 1) / TG;
  const int64_t waves = int64_t(p.units) * ngroups;
  const int64_t blocks = (waves + kWaves - 1) / kWaves;
  if (blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((prompt_valu_kernel<ES, D, G>), dim3(unsigned(blocks)), dim3(kThreads), 0, s,
                     p, ngroups);
  return hipGetLastError();
}

template <int ES, int D>
hipError_t prompt_by_group(int group, bool vt, const PromptParams &p, const Control *ctrl,
                           hipStream_t s) {
  (void)ctrl;
  if constexpr (ES == 2) {
    switch (group) {
      case 1: return prompt_mfma<D, 1>(p, vt, s);
      case 2: return prompt_mfma<D, 2>(p, vt, s);
      case 4: return prompt_mfma<D, 4>(p, vt, s);
      case 8: return prompt_mfma<D, 8>(p, vt, s);
      default: return hipErrorInvalidValue;
    }
  } else {
    (void)vt;
    switch (group) {
      case 1: return prompt_valu<ES, D, 1>(p, s);
      case 2: return prompt_valu<ES, D, 2>(p, s);
      case 4: return prompt_valu<ES, D, 4>(p, s);
      case 8: return prompt_valu<ES, D, 8>(p, s);
      default: return hipErrorInvalidValue;
    }
  }
}

}  // namespace

hipError_t launch_prompt_attend(int elem_bytes, int head_dim, int group, bool vt,
                                const PromptParams &p, const Control *ctrl, hipStream_t s) {
  if (p.n == 0) return hipSuccess;
  if (elem_bytes == 2)
    return head_dim == 128 ? prompt_by_group<2, 128>(group, vt, p, ctrl, s)
                           : prompt_by_group<2, 64>(group, vt, p, ctrl, s);
  return head_dim == 128 ? prompt_by_group<4, 128>(group, vt, p, ctrl, s)
                         : prompt_by_group<4, 64>(group, vt, p, ctrl, s);
}

}  // namespace dmc
