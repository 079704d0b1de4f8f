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
#include "dmc_device.h"

namespace dmc {
namespace {

// Orders this wave's LDS writes before its later LDS reads (and the reverse).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

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

// ---------------------------------------------------------------------------
// bf16 on matrix cores.  One workgroup = 4 waves = one unit's 128 query
// columns (token-major: column c is token c / G, head c % G of the group);
// each wave owns 32 columns, T = 32 / G tokens.  The unit's closed slots
// stream through LDS in blocks of 32, shared by the 4 waves; per block and
// wave
//   S^T[slot][col]  = K[slot][:] . Q[col][:]          (A = K, B = Q^T)
//   O^T[dim][col]  += V^T[dim][slot] P^T[slot][col]    (A = V^T, B = P^T)
// on v_mfma_f32_16x16x32_bf16, with the interleaved key-row assignment of
// the decode kernel (score tile sb, row m -> block slot 8(m/4) + 4 sb + m%4)
// so that the score tile's output registers are already the P^T operand.
//
// Blocks arrive by direct global -> LDS transfers (16 bytes per lane, no
// registers) into a ring of kStages buffers, kStages - 1 blocks ahead of the
// one being multiplied.  Key rows land XOR-swizzled in 16-byte units so that
// each 16-lane group's operand loads hit distinct banks.  Value rows are
// read transposed by ds_read_b64_tr_b16 (a 16-lane group pointing at four
// 8-byte row pieces each of 4 rows receives, per lane, one column's 4
// consecutive rows); caches that store value pages transposed ([d][P]) are
// read as V^T rows directly.  Workgroups are mapped so that all tiles of a
// unit run on one XCD (sharing its L2), latest tiles (most slots) first.  P
// enters the value product rounded to bf16 and its sum is taken over the
// rounded values.
// ---------------------------------------------------------------------------
#ifndef DMC_PROMPT_STAGES
#define DMC_PROMPT_STAGES 3
#endif
constexpr int kStages = DMC_PROMPT_STAGES;
constexpr int kPtabLds = kPromptMaxPages;   // page-table entries of a unit cached in LDS

template <int CPR>
__device__ __forceinline__ int k_swizzle(int row) {   // physical 16-byte chunk = logical ^ this
  return ((row & 3) | (((row >> 3) & 3) << 2)) & (CPR - 1);
}
template <int CPR>
__device__ __forceinline__ int v_swizzle(int row) { return (2 * (row & 3)) & (CPR - 1); }
__device__ __forceinline__ int vt_swizzle(int dim) { return (dim >> 2) & 3; }

__device__ __forceinline__ uint32_t lds_offset(const void *p) {
  return static_cast<uint32_t>(
      reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const char *)p));
}

// 16 bytes per lane from global memory straight into LDS at
// lds_base + 16 * lane (lds_base wave-uniform).  Issued as inline assembly so
// that the compiler neither waits for it nor reorders LDS accesses around it;
// completion is awaited with wait_vmcnt before the workgroup barrier.
__device__ __forceinline__ void dma16(uint32_t lds_base, const void *g) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(lds_base), "v"(g)
               : "memory");
}

// s_waitcnt with only the vector-memory count (at most N outstanding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;

__device__ __forceinline__ uint2 ds_read_tr16(const void *p) {
  const bf16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (lds_bf16x4_t *)((__attribute__((address_space(3))) char *)p));
  return __builtin_bit_cast(uint2, v);
}

// Two floats -> packed bf16 pair (round to nearest even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
  typedef float f2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 b2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f2_t{lo, hi}, b2_t));
}

template <int D, int G, bool VT>
__global__ __launch_bounds__(kThreads, 2) void prompt_mfma_kernel(PromptParams p, int ntiles) {
  constexpr int T = 32 / G;            // tokens per wave
  constexpr int TW = kWaves * T;       // tokens per workgroup
  constexpr int KS = D / 32, NT = D / 16, RB = D * 2;
  constexpr int CPR = D / 8;           // 16-byte chunks per row
  constexpr int BLK = 32 * RB;         // bytes of one block's keys (and of its values)
  constexpr int DPW = BLK / 16 / kThreads;   // transfers per thread per block half
  constexpr int SBYTES = kStages * 2 * BLK;
  constexpr int STAGE = 8 * 2 * D;     // floats per wave: 8 tokens x (key mean, value mean)
  static_assert(kWaves * STAGE * 4 <= SBYTES, "open-state staging fits the block ring");
  static_assert(DPW >= 1 && BLK % (16 * kThreads) == 0, "block split");
  static_assert(kStages >= 2 && kStages <= 4, "ring depth");
  __shared__ __align__(16) unsigned char smem[SBYTES];
  __shared__ int s_hi[kWaves];
  __shared__ int s_pt[kPtabLds];

  const int bid = blockIdx.x;
  const int xcd = bid & 7, r = bid >> 3;
  const int ul = r / ntiles, tile = ntiles - 1 - (r - ul * ntiles);
  const int u = ul * 8 + xcd;
  if (u >= p.units) return;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n16 = lane & 15, q4 = lane >> 4;
  const int b = u / p.hkv, g = u - b * p.hkv;
  const int nb = clamp_prompt_len(p.prompt_lens, p.n, b);
  const bool ok = p.page_base[u] >= 0;
  const int a = tile * TW + wave * T;
  const int cnt = ok ? max(0, min(T, nb - a)) : 0;
  const uint4 zero4 = make_uint4(0, 0, 0, 0);

  const int seg = cnt > 0 ? token_slots(p, u, a, cnt) : -1;
  int lim[2], tok[2];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    tok[qb] = (16 * qb + n16) / G;
    const int sj = __shfl(seg, tok[qb], 64);
    lim[qb] = tok[qb] < cnt ? sj : 0;
  }
  const int wave_hi = cnt > 0 ? __shfl(seg, cnt - 1, 64) : 0;
  if (lane == 0) s_hi[wave] = wave_hi;

  // Q^T operand: lane (n16, q4) holds Q[col 16 qb + n16][32 ks + 8 q4 .. +8].
  uint4 qop[2][KS];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    const int j = tok[qb], h = 16 * qb + n16 - j * G;
    const char *qr = static_cast<const char *>(p.q) +
                     (b * p.qs[0] + int64_t(a + j) * p.qs[1] + (g * G + h) * p.qs[2]) * 2;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qop[qb][ks] = j < cnt ? ld16(qr + ks * 64 + q4 * 16) : zero4;
    if (q4 == 0) qop[qb][0].x &= 0xffff0000u;   // q[0] is not part of the score
  }

  float m[2] = {0.0f, 0.0f}, ls[2] = {0.0f, 0.0f};
  f32x4_t acc[2][NT];
#pragma unroll
  for (int qb = 0; qb < 2; ++qb)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[qb][nt] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

  // Open state of each column's token.  The walk stages key and value means
  // of 8 tokens at a time (fp32, this wave's part of the block ring); then
  // every lane takes its columns' score (dot with its Q^T slice, summed over
  // the 4 lane groups) and its slice of the value mean.
  if (cnt > 0) {
    float *stage = reinterpret_cast<float *>(smem) + wave * STAGE;
    constexpr int E = D / 64;
    walk_open_state<2, D>(
        p, u, b, g, a, cnt,
        [&](int t, const float *ak, const float *av, float zs) {
          const float inv = 1.0f / zs;
          float *row = stage + (t & 7) * 2 * D;
#pragma unroll
          for (int e = 0; e < E; ++e) {
            row[lane * E + e] = ak[e] * inv;
            row[D + lane * E + e] = av[e] * inv;
          }
        },
        [&](int t0) {
          if (t0 + 8 <= a) return;   // nothing staged in this batch
          wave_lds_sync();
          float part[2];
          bool here[2];
#pragma unroll
          for (int qb = 0; qb < 2; ++qb) {
            const int t = a + tok[qb];
            here[qb] = tok[qb] < cnt && t >= t0 && t < t0 + 8;
            part[qb] = 0.0f;
            if (here[qb]) {
              const float *kp = stage + (t & 7) * 2 * D;
#pragma unroll
              for (int ks = 0; ks < KS; ++ks) {
                float qf[8];
                V16<2>::unpack(qop[qb][ks], qf);
                const float4 k0 = *reinterpret_cast<const float4 *>(kp + 32 * ks + 8 * q4);
                const float4 k1 = *reinterpret_cast<const float4 *>(kp + 32 * ks + 8 * q4 + 4);
                part[qb] = fmaf(qf[0], k0.x, part[qb]);
                part[qb] = fmaf(qf[1], k0.y, part[qb]);
                part[qb] = fmaf(qf[2], k0.z, part[qb]);
                part[qb] = fmaf(qf[3], k0.w, part[qb]);
                part[qb] = fmaf(qf[4], k1.x, part[qb]);
                part[qb] = fmaf(qf[5], k1.y, part[qb]);
                part[qb] = fmaf(qf[6], k1.z, part[qb]);
                part[qb] = fmaf(qf[7], k1.w, part[qb]);
              }
            }
          }
#pragma unroll
          for (int qb = 0; qb < 2; ++qb) {
            part[qb] += __shfl_xor(part[qb], 16, 64);
            part[qb] += __shfl_xor(part[qb], 32, 64);
          }
#pragma unroll
          for (int qb = 0; qb < 2; ++qb) {
            if (here[qb]) {
              const float *vp = stage + ((a + tok[qb]) & 7) * 2 * D + D;
              m[qb] = part[qb] * p.scale_log2;
              ls[qb] = q4 == 0 ? 1.0f : 0.0f;   // the open state's weight, counted once
#pragma unroll
              for (int nt = 0; nt < NT; ++nt) {
                const float4 x = *reinterpret_cast<const float4 *>(vp + 16 * nt + 4 * q4);
                acc[qb][nt] = f32x4_t{x.x, x.y, x.z, x.w};
              }
            }
          }
          wave_lds_sync();
        });
  }
  __syncthreads();   // slot limits published; staging area free again

  int s_top = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) s_top = max(s_top, s_hi[w]);
  const int nblk = (s_top + 31) >> 5;
  const int P = 1 << p.log2p;
  const int64_t pt = int64_t(u) * p.maxpages;
  const int npg = min((s_top + P - 1) >> p.log2p, kPtabLds);
  for (int i = tid; i < npg; i += kThreads) s_pt[i] = p.ptab[pt + i];
  __syncthreads();
  // The host limits this kernel to prompts of at most kPtabLds pages per unit.
  auto page_of = [&](int s) -> const char * {
    return p.pool + int64_t(s_pt[s >> p.log2p]) * p.page_bytes;
  };

  // Transfers of block kb into ring slot st; rows past the closed slots read
  // the last closed one (in bounds; masked or zeroed when used).
  const uint32_t ring = lds_offset(smem);
  auto issue = [&](int kb, int st) {
#pragma unroll
    for (int i = 0; i < DPW; ++i) {
      const int run = i * kWaves + wave;   // 1 KB run of the block written by this instruction
      const int c = run * 64 + lane;       // 16-byte chunk of the block
      const uint32_t kdst = __builtin_amdgcn_readfirstlane(ring + st * 2 * BLK + run * 1024);
      const int row = c / CPR, pc = c - row * CPR;
      const int s = min(kb * 32 + row, s_top - 1);
      const char *krow = page_of(s) + int64_t(s & (P - 1)) * RB;
      dma16(kdst, krow + (pc ^ k_swizzle<CPR>(row)) * 16);
      const char *gv;
      if (VT) {   // value page [D][P]: chunk = (dim, 8 slots)
        const int dim = c >> 2, lc = (c & 3) ^ vt_swizzle(dim);
        const int s0 = min(kb * 32 + 8 * lc, (s_top - 1) & ~7);
        gv = page_of(s0) + int64_t(P) * RB + (int64_t(dim) * P + (s0 & (P - 1))) * 2;
      } else {
        gv = krow + int64_t(P) * RB + (pc ^ v_swizzle<CPR>(row)) * 16;
      }
      dma16(kdst + BLK, gv);
    }
  };

  for (int kb = 0; kb < kStages - 1 && kb < nblk; ++kb) issue(kb, kb);
  const int krow0 = 8 * (n16 >> 2) + (n16 & 3);   // score tile 0 row of this lane (+4 in tile 1)
  for (int kb = 0; kb < nblk; ++kb) {
    // blocks issued after kb: min(nblk - 1 - kb, kStages - 2)
    const int after = min(nblk - 1 - kb, kStages - 2);
    if (after >= 2) wait_vmcnt<4 * DPW>();
    else if (after == 1) wait_vmcnt<2 * DPW>();
    else wait_vmcnt<0>();
    __syncthreads();   // block kb is in LDS for every wave; the ring slot of kb - 1 is free
    if (kb + kStages - 1 < nblk) issue(kb + kStages - 1, (kb + kStages - 1) % kStages);
    if (kb * 32 >= wave_hi) continue;
    const int st = kb % kStages;
    const char *kd = reinterpret_cast<const char *>(smem) + st * 2 * BLK;
    const char *vd = kd + BLK;
    f32x4_t sc[2][2];
#pragma unroll
    for (int sb = 0; sb < 2; ++sb)
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) sc[sb][qb] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      uint4 ka[2];
#pragma unroll
      for (int sb = 0; sb < 2; ++sb) {
        const int row = krow0 + 4 * sb;
        ka[sb] = *reinterpret_cast<const uint4 *>(kd + row * RB +
                                                  (((4 * ks + q4) ^ k_swizzle<CPR>(row)) * 16));
      }
#pragma unroll
      for (int sb = 0; sb < 2; ++sb)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) sc[sb][qb] = mfma_16x16x32(ka[sb], qop[qb][ks], sc[sb][qb]);
    }
    // V^T operands of the value product: lane (n16, q4) = dim 16 nt + n16, slots 8 q4 .. +8.
    uint4 va[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      if (VT) {
        const int dim = 16 * nt + n16;
        va[nt] = *reinterpret_cast<const uint4 *>(vd + dim * 64 + ((q4 ^ vt_swizzle(dim)) * 16));
      } else {
        uint2 h[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int row = 8 * q4 + 4 * hh + (n16 >> 2);
          const int lc = 2 * nt + ((n16 & 3) >> 1);
          h[hh] = ds_read_tr16(vd + row * RB + ((lc ^ v_swizzle<CPR>(row)) * 16) + (n16 & 1) * 8);
        }
        va[nt] = make_uint4(h[0].x, h[0].y, h[1].x, h[1].y);
      }
    }
    const int keep = s_top - (kb * 32 + 8 * q4);   // this lane's slots below s_top
    if (keep < 8) {
      uint32_t msk[4];
#pragma unroll
      for (int w = 0; w < 4; ++w)
        msk[w] = (2 * w < keep ? 0x0000ffffu : 0u) | (2 * w + 1 < keep ? 0xffff0000u : 0u);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        va[nt].x &= msk[0];
        va[nt].y &= msk[1];
        va[nt].z &= msk[2];
        va[nt].w &= msk[3];
      }
    }
    uint4 pb[2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      float x[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int s = kb * 32 + 8 * q4 + j;
        x[j] = s < lim[qb] ? sc[j >> 2][qb][j & 3] * p.scale_log2 : neg_inf();
      }
      float mx = x[0];
#pragma unroll
      for (int j = 1; j < 8; ++j) mx = fmaxf(mx, x[j]);
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mn = fmaxf(m[qb], mx);
      const float f = fast_exp2(m[qb] - mn);
      m[qb] = mn;
      ls[qb] *= f;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) acc[qb][nt] *= f;
      uint32_t pw[4];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        pw[w] = cvt_pk_bf16(fast_exp2(x[2 * w] - mn), fast_exp2(x[2 * w + 1] - mn));
        ls[qb] += __uint_as_float(pw[w] << 16) + __uint_as_float(pw[w] & 0xffff0000u);
      }
      pb[qb] = make_uint4(pw[0], pw[1], pw[2], pw[3]);
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int qb = 0; qb < 2; ++qb) acc[qb][nt] = mfma_16x16x32(va[nt], pb[qb], acc[qb][nt]);
  }

  // Normalise and store: lane holds dims 16 nt + 4 q4 .. +4 of its columns.
#pragma unroll
  for (int qb = 0; qb < 2; ++qb) {
    float lt = ls[qb];
    lt += __shfl_xor(lt, 16, 64);
    lt += __shfl_xor(lt, 32, 64);
    const int j = tok[qb], h = 16 * qb + n16 - j * G;
    const int t = a + j;
    if (t >= p.n) continue;
    const bool valid = j < cnt;
    const float inv = valid ? 1.0f / lt : 0.0f;
    char *orow = static_cast<char *>(p.out) +
                 (b * p.os[0] + int64_t(t) * p.os[1] + (g * G + h) * p.os[2]) * 2;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const uint32_t lo = cvt_pk_bf16(acc[qb][nt][0] * inv, acc[qb][nt][1] * inv);
      const uint32_t hi = cvt_pk_bf16(acc[qb][nt][2] * inv, acc[qb][nt][3] * inv);
      *reinterpret_cast<uint2 *>(orow + (16 * nt + 4 * q4) * 2) = make_uint2(lo, hi);
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
    walk_open_state<ES, D>(
        p, u, b, g, a, cnt,
        [&](int t, const float *ak, const float *av, float zs) {
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
        },
        [](int) {});
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
    hipLaunchKernelGGL((prompt_mfma_kernel<D, G, true>), dim3(unsigned(blocks)), dim3(kThreads), 0,
                       s, p, ntiles);
  else
    hipLaunchKernelGGL((prompt_mfma_kernel<D, G, false>), dim3(unsigned(blocks)), dim3(kThreads), 0,
                       s, p, ntiles);
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
