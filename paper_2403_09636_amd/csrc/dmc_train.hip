// gfx950 kernels of DMC's training-time forward and backward.
//
// Method: Nawrot et al., "Dynamic Memory Compression" (ICML 2024), Sec. 3.2
// (Training), Sec. 3.3 (window grouping) and the masking appendix:
//   alpha_t = sigmoid(x_t), x_t = (k_t[0] - c + g_t) / tau   (Gumbel-sigmoid,
//             logistic noise g supplied by the caller),
//   omega_t = sigmoid(q_t[lead][0])  (or 1: uniform weighting),
//   state j = partial accumulation over tokens a_j = max(0, j - w + 1) .. j:
//             K~_j = sum_t c_tj k^_t / z_j, c_tj = omega_t prod_{r=t+1..j} alpha_r,
//             z_j = sum_t c_tj (the recurrence of Sec. 3.2 in closed form; the
//             window's first token enters with weight omega alone),
//   scores   q_i[1:] . K~_j[1:] / sqrt(d) + M_ij, M_ij = log(1 - alpha_{j+1})
//             = log-sigmoid(-x_{j+1}) for j < i, 0 for j = i, -inf for j > i.
//
// Forward: per-token decisions and mask, the unrolled states, then masked
// softmax attention (softmax statistics kept for the backward).  Backward:
// dq per query row; dK~, dV~ and the mask gradient per state; then the
// states' gradients are carried back to the tokens (the closed form above),
// and the decision / importance neurons get theirs through alpha and omega.
//
// Vector-ALU kernels (lanes own head-dim elements, one wave per group of
// rows) serve every dtype; bf16 attention runs on the matrix cores
// (v_mfma_f32_32x32x16_bf16) in four kernels: forward, dq, dV~, and dK~ with
// the mask gradient.
#include <type_traits>

#include "dmc_mfma.h"

namespace dmc {

TrainLayout train_layout(int batch, int n, int hq, int hkv, int head_dim, int elem_bytes,
                         int window) {
  TrainLayout L{};
  const size_t U = size_t(batch) * hkv, G = size_t(hq / hkv), N = size_t(n), D = head_dim;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes, 256);
    return at;
  };
  // states: 32 rows of (zeroed) padding so that 32-row blocks never leave the buffer
  L.ks = take((U * N + 32) * D * elem_bytes);
  L.vs = take((U * N + 32) * D * elem_bytes);
  L.alpha = take(U * N * 4);
  L.omega = take(U * N * 4);
  L.z = take(U * N * 4);
  L.mask = take(U * N * 4);
  L.lse = take((U * G * N + 32) * 4);   // [U][n][G], padded for 32-row statistics transfers
  L.dsum = take((U * G * N + 32) * 4);
  L.dks = take(U * N * D * 4);
  L.dvs = take(U * N * D * 4);
  L.dmask = take(U * N * 4);
  L.qs = take(2 * U * N * 4);
  L.e = take(U * N * size_t(window) * 4);
  L.total = off;
  return L;
}

namespace {

constexpr float kLog2e = 1.4426950408889634f;


// log(1 - sigmoid(x)) = -softplus(x), without cancellation.
__device__ __forceinline__ float log_one_minus_sigmoid(float x) {
  return -(fmaxf(x, 0.0f) + log1pf(expf(-fabsf(x))));
}

__device__ __forceinline__ float wsum(float x) {
  x = row_sum<32>(x);
  return x + __shfl_xor(x, 32, 64);
}

// Row offsets (elements) of the [B, n, H, d] tensors.
__device__ __forceinline__ int64_t row_q(const TrainParams &p, int b, int t, int h, int D) {
  return ((int64_t(b) * p.n + t) * p.hq + h) * D;
}
__device__ __forceinline__ int64_t row_k(const TrainParams &p, int b, int t, int g, int D) {
  return ((int64_t(b) * p.n + t) * p.hkv + g) * D;
}

// Per token: alpha and omega from the Gumbel-sigmoid logit and the query
// neuron; the mask entry of the previous state (log(1 - alpha_t) belongs to
// state t - 1).
template <int ES, int D>
__global__ __launch_bounds__(kThreads) void train_decide_kernel(TrainParams p) {
  const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  const int U = p.batch * p.hkv;
  if (i >= int64_t(U) * p.n) return;
  const int u = static_cast<int>(i / p.n), t = static_cast<int>(i - int64_t(u) * p.n);
  const int b = u / p.hkv, g = u - b * p.hkv, G = p.hq / p.hkv;
  const float k0 = load_elem<ES>(p.k, row_k(p, b, t, g, D));
  const float g_noise = p.noise[(int64_t(b) * p.n + t) * p.hkv + g];
  const float x = (k0 - p.c + g_noise) / p.tau;
  const float al = 1.0f / (1.0f + expf(-x));
  float om = 1.0f;
  if (p.omega_src == 0) om = sigmoid_floor(load_elem<ES>(p.q, row_q(p, b, t, g * G, D)));
  p.alpha[i] = al;
  p.omega[i] = om;
  if (p.alpha_out) p.alpha_out[(int64_t(b) * p.n + t) * p.hkv + g] = al;
  if (t > 0) p.mask[i - 1] = log_one_minus_sigmoid(x);
  if (t == p.n - 1) p.mask[i] = 0.0f;   // the last state has no successor
}

// Unrolled states, one wave per (unit, 64 positions), NP positions at a
// time: state j is the closed-form partial accumulation over its window,
// summed from token j down to the window start with the running product of
// alphas.  The NP positions share their tokens' rows, which are loaded in
// batches and added to every position whose window holds them (each
// position's sum runs over its tokens in the same descending order).
template <int ES, int D>
__global__ __launch_bounds__(64) void train_states_kernel(TrainParams p) {
  constexpr int E = D / 64, NP = 8, kB = 8;
  const int u = blockIdx.y, lane = threadIdx.x;
  const int b = u / p.hkv, g = u - b * p.hkv;
  const int j0 = blockIdx.x * 64, j1 = min(j0 + 64, p.n);
  const float *al = p.alpha + int64_t(u) * p.n;
  const float *om = p.omega + int64_t(u) * p.n;
  const char *kb = static_cast<const char *>(p.k) + (row_k(p, b, 0, g, D) + lane * E) * ES;
  const char *vb = static_cast<const char *>(p.v) + (row_k(p, b, 0, g, D) + lane * E) * ES;
  const int64_t rs = int64_t(p.hkv) * D * ES;   // bytes between tokens
  const float sqrt_d = kLog2e / p.scale_log2;
  for (int jg = j0; jg < j1; jg += NP) {
    const int np = min(NP, j1 - jg);
    const int jl = jg + np - 1;                   // last position of the group
    const int lo = max(0, jg - p.window + 1);     // first token any of them needs
    float sk[NP][E], sv[NP][E], zs[NP], P[NP];
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      zs[i] = 0.0f;
      P[i] = 1.0f;
#pragma unroll
      for (int e = 0; e < E; ++e) sk[i][e] = sv[i][e] = 0.0f;
    }
    for (int t0 = jl; t0 >= lo; t0 -= kB) {
      float kk[kB][E], vv[kB][E], wa[kB], wo[kB];
#pragma unroll
      for (int q = 0; q < kB; ++q) {
        const int t = max(t0 - q, lo);
        load_e<ES, E>(kb + t * rs, kk[q]);
        load_e<ES, E>(vb + t * rs, vv[q]);
        wa[q] = al[t];
        wo[q] = om[t];
      }
#pragma unroll
      for (int q = 0; q < kB; ++q) {
        const int t = t0 - q;
        if (t < lo) break;
        if (lane == 0) kk[q][0] = 0.0f;   // k_t[0] <- 0
#pragma unroll
        for (int i = 0; i < NP; ++i) {
          const int j = jg + i;
          if (i >= np || t > j || t < j - p.window + 1) continue;
          const float c = wo[q] * P[i];    // omega_t * prod_{r = t+1 .. j} alpha_r
#pragma unroll
          for (int e = 0; e < E; ++e) {
            sk[i][e] = fmaf(c, kk[q][e], sk[i][e]);
            sv[i][e] = fmaf(c, vv[q][e], sv[i][e]);
          }
          zs[i] += c;
          P[i] *= wa[q];
        }
      }
    }
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      if (i >= np) break;
      const int j = jg + i;
      const float inv = 1.0f / zs[i];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        sk[i][e] *= inv;
        sv[i][e] *= inv;
      }
      // Element 0 of a key state is never part of a score; it carries the
      // state's mask entry times sqrt(d), which the matrix-core kernels add
      // to the scores through a query element fixed at 1.
      if (lane == 0) sk[i][0] = p.mask[int64_t(u) * p.n + j] * sqrt_d;
      const int64_t o = (int64_t(u) * p.n + j) * D + lane * E;
      store_e<ES, E>(static_cast<char *>(p.ks) + o * ES, sk[i]);
      store_e<ES, E>(static_cast<char *>(p.vs) + o * ES, sv[i]);
      if (lane == 0) p.z[int64_t(u) * p.n + j] = zs[i];
    }
  }
}

// Unrolled states on the matrix cores (bf16), one wave per (unit, 32
// positions j0 .. j0 + 31).  The wave stages the raw key and value rows of
// tokens tb = j0 - 16 (NK - 2) .. j0 + 31 in LDS (direct transfers, value
// swizzle) and forms, per position (lane column), the closed-form weights
// c_tj = omega_t prod_{r=t+1..j} alpha_r of its window in registers, walking
// the tokens downwards from j exactly as the vector kernel does (so z_j is
// the same fp32 sum).  Then, per 32-dim tile,
//   S^T[dim][j] = sum_t K^T[dim][t] C^T[t][j]   (A: transposed LDS reads,
//                                                B: the lane's weights)
// with each weight split into a bf16 head and tail (c = hi + lo to about
// 2^-17 relative), and the same for the values.  NK 16-token k-steps cover
// the 31 + w tokens that the 32 positions need.
template <int D, int NK>
__global__ __launch_bounds__(64) void train_states_mfma_kernel(TrainParams p) {
  constexpr int RB = D * 2, CPR = D / 8, NTL = D / 32, ROWS = 16 * NK;
  constexpr int NDMA = ROWS * CPR / 64;   // 16-byte transfers per lane and matrix
  static_assert(ROWS * CPR % 64 == 0, "row staging split");
  __shared__ __align__(16) unsigned char smem[2 * ROWS * RB];
  const int u = blockIdx.y, lane = threadIdx.x;
  const int col = lane & 31, hb = lane >> 5;
  const int b = u / p.hkv, g = u - b * p.hkv;
  const int j0 = blockIdx.x * 32;
  const int tb = j0 - 16 * (NK - 2);
  const int W = p.window, last = p.n - 1;

  // Raw rows of tokens tb .. tb + ROWS - 1 (clamped into the sequence; the
  // rows outside it get weight 0).
  const char *kb = static_cast<const char *>(p.k) + row_k(p, b, 0, g, D) * 2;
  const char *vb = static_cast<const char *>(p.v) + row_k(p, b, 0, g, D) * 2;
  const int64_t rs = int64_t(p.hkv) * D * 2;
#pragma unroll
  for (int i = 0; i < NDMA; ++i) {
    const int c = i * 64 + lane;
    const int row = c / CPR, pc = c - row * CPR;
    const int64_t src = min(max(tb + row, 0), last) * rs + (pc ^ v_swizzle<CPR>(row)) * 16;
    dma16(smem + i * 1024, kb + src);
    dma16(smem + ROWS * RB + i * 1024, vb + src);
  }

  // Weights of position j for staged rows 0 .. ROWS - 1, from the top down.
  const float *al = p.alpha + int64_t(u) * p.n;
  const float *om = p.omega + int64_t(u) * p.n;
  const int j = j0 + col;
  float cw[ROWS];
  float zs = 0.0f, P = 1.0f;
#pragma unroll
  for (int r = ROWS - 1; r >= 0; --r) {
    const int t = tb + r;
    const int tc = min(max(t, 0), last);
    const float a = al[tc], o = om[tc];
    const bool in = t <= j && t > j - W && t >= 0;
    const float c = in ? o * P : 0.0f;
    cw[r] = c;
    zs += c;
    if (in) P *= a;
  }
  // This lane's half (rows 16 ks + 8 hb + e) as packed bf16 head and tail.
  uint4 whi[NK], wlo[NK];
#pragma unroll
  for (int ks = 0; ks < NK; ++ks) {
    uint32_t h[4], l[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float w0 = hb ? cw[16 * ks + 8 + 2 * q] : cw[16 * ks + 2 * q];
      const float w1 = hb ? cw[16 * ks + 9 + 2 * q] : cw[16 * ks + 1 + 2 * q];
      h[q] = cvt_pk_bf16(w0, w1);
      l[q] = cvt_pk_bf16(w0 - __uint_as_float(h[q] << 16), w1 - __uint_as_float(h[q] & 0xffff0000u));
    }
    whi[ks] = make_uint4(h[0], h[1], h[2], h[3]);
    wlo[ks] = make_uint4(l[0], l[1], l[2], l[3]);
  }

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
  wait_vmcnt<0>();
  wave_lds_sync();

  const float inv = 1.0f / zs;
  const float sqrt_d = kLog2e / p.scale_log2;
  if (j < p.n && hb == 0) p.z[int64_t(u) * p.n + j] = zs;
  const float mask_j = j < p.n ? p.mask[int64_t(u) * p.n + j] * sqrt_d : 0.0f;
  const int nrow = min(32, p.n - j0);   // positions of this block inside the sequence
#pragma unroll
  for (int m = 0; m < 2; ++m) {
    char *buf = reinterpret_cast<char *>(smem) + m * ROWS * RB;
    f32x16_t acc[NTL];
#pragma unroll
    for (int t = 0; t < NTL; ++t) {
      acc[t] = f32x16_t{};
#pragma unroll
      for (int ks = 0; ks < NK; ++ks) {
        const uint2 h0 = ds_read_tr16(buf + vaddr[t] + 16 * ks * RB);
        const uint2 h1 = ds_read_tr16(buf + vaddr[t] + (16 * ks + 4) * RB);
        const uint4 a = make_uint4(h0.x, h0.y, h1.x, h1.y);
        acc[t] = mfma_32x32x16(a, whi[ks], acc[t]);
        acc[t] = mfma_32x32x16(a, wlo[ks], acc[t]);
      }
    }
    // The 32 state rows back into this matrix's staging rows 0 .. 31 (its
    // inputs are consumed), 16-byte chunks XOR-swizzled by row; lane holds
    // dims 32 t + 8 i + 4 hb .. + 4 of position j0 + col.
#pragma unroll
    for (int t = 0; t < NTL; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float x0 = acc[t][4 * i] * inv;
        if (m == 0 && t == 0 && i == 0 && hb == 0) x0 = mask_j;   // the mask carrier
        const uint32_t lo = cvt_pk_bf16(x0, acc[t][4 * i + 1] * inv);
        const uint32_t hi = cvt_pk_bf16(acc[t][4 * i + 2] * inv, acc[t][4 * i + 3] * inv);
        *reinterpret_cast<uint2 *>(buf + col * RB + (((4 * t + i) ^ k_swizzle<CPR>(col)) * 16) + hb * 8) =
            make_uint2(lo, hi);
      }
    wave_lds_sync();
    // Whole rows out: 64 / CPR rows per pass, 16 bytes per lane.
    char *dst = static_cast<char *>(m == 0 ? p.ks : p.vs) + (int64_t(u) * p.n + j0) * RB;
    constexpr int RPP = 64 / CPR;
#pragma unroll
    for (int r0 = 0; r0 < 32; r0 += RPP) {
      const int row = r0 + lane / CPR, ch = lane % CPR;
      if (row < nrow)
        *reinterpret_cast<uint4 *>(dst + row * RB + ch * 16) =
            *reinterpret_cast<const uint4 *>(buf + row * RB + ((ch ^ k_swizzle<CPR>(row)) * 16));
    }
  }
}

// Rows handled by one wave of the attention kernels: TG tokens x G heads.
template <int G>
struct Rows {
  static constexpr int TG = G >= 8 ? 1 : 8 / G;
  static constexpr int R = TG * G;
};

// Forward attention over the states: one wave per (unit, TG tokens), row r =
// token a + r / G, head r % G; online softmax in the log2 domain.
template <int ES, int D, int G>
__global__ __launch_bounds__(kThreads) void train_fwd_kernel(TrainParams p, int ngroups) {
  constexpr int TG = Rows<G>::TG, R = Rows<G>::R, E = D / 64, kAhead = 4;
  const int lane = threadIdx.x & 63;
  const int wid = blockIdx.x * kWaves + (threadIdx.x >> 6);
  const int U = p.batch * p.hkv;
  const int u = wid / ngroups;
  if (u >= U) return;
  const int a = (wid - u * ngroups) * TG;
  const int cnt = min(TG, p.n - a);
  const int b = u / p.hkv, g = u - b * p.hkv;
  float qr[R][E];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j = r / G, h = r - j * G;
#pragma unroll
    for (int e = 0; e < E; ++e) qr[r][e] = 0.0f;
    if (j < cnt)
      load_e<ES, E>(static_cast<const char *>(p.q) + (row_q(p, b, a + j, g * G + h, D) + lane * E) * ES,
                    qr[r]);
    if (lane == 0) qr[r][0] = 0.0f;   // q[0] is not part of the score
  }
  float m[R], l[R], acc[R][E];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    m[r] = neg_inf();
    l[r] = 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) acc[r][e] = 0.0f;
  }
  const int last = a + cnt - 1;
  const char *ksb = static_cast<const char *>(p.ks) + (int64_t(u) * p.n * D + lane * E) * ES;
  const char *vsb = static_cast<const char *>(p.vs) + (int64_t(u) * p.n * D + lane * E) * ES;
  const float *mk = p.mask + int64_t(u) * p.n;
  for (int s0 = 0; s0 <= last; s0 += kAhead) {
    float kk[kAhead][E], vv[kAhead][E], bias[kAhead];
#pragma unroll
    for (int i = 0; i < kAhead; ++i) {
      const int s = min(s0 + i, last);
      load_e<ES, E>(ksb + int64_t(s) * D * ES, kk[i]);
      load_e<ES, E>(vsb + int64_t(s) * D * ES, vv[i]);
      bias[i] = mk[s] * kLog2e;
    }
#pragma unroll
    for (int i = 0; i < kAhead; ++i) {
      const int s = s0 + i;
      if (s > last) break;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int t = a + r / G;
        if (r / G >= cnt || s > t) continue;
        float d = 0.0f;
#pragma unroll
        for (int e = 0; e < E; ++e) d = fmaf(qr[r][e], kk[i][e], d);
        const float x = wsum(d) * p.scale_log2 + (s < t ? bias[i] : 0.0f);
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
    if (j >= cnt) continue;
    float o[E];
    const float inv = 1.0f / l[r];
#pragma unroll
    for (int e = 0; e < E; ++e) o[e] = acc[r][e] * inv;
    store_e<ES, E>(static_cast<char *>(p.out) + (row_q(p, b, a + j, g * G + h, D) + lane * E) * ES, o);
    if (lane == 0) p.lse[(int64_t(u) * p.n + a + j) * G + h] = m[r] + __log2f(l[r]);
  }
}

// dq of every query row, and D = sum(dout * out) of the row for the state
// kernel: one wave per (unit, TG tokens), keys streamed as in the forward.
template <int ES, int D, int G>
__global__ __launch_bounds__(kThreads) void train_dq_kernel(TrainParams p, int ngroups) {
  constexpr int TG = Rows<G>::TG, R = Rows<G>::R, E = D / 64, kAhead = 4;
  const int lane = threadIdx.x & 63;
  const int wid = blockIdx.x * kWaves + (threadIdx.x >> 6);
  const int U = p.batch * p.hkv;
  const int u = wid / ngroups;
  if (u >= U) return;
  const int a = (wid - u * ngroups) * TG;
  const int cnt = min(TG, p.n - a);
  const int b = u / p.hkv, g = u - b * p.hkv;
  float qr[R][E], dor[R][E], Lr[R], Dr[R], dq[R][E];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j = r / G, h = r - j * G;
#pragma unroll
    for (int e = 0; e < E; ++e) qr[r][e] = dor[r][e] = dq[r][e] = 0.0f;
    Lr[r] = 0.0f;
    Dr[r] = 0.0f;
    if (j < cnt) {
      const int64_t ro = row_q(p, b, a + j, g * G + h, D) + lane * E;
      float of[E];
      load_e<ES, E>(static_cast<const char *>(p.q) + ro * ES, qr[r]);
      load_e<ES, E>(static_cast<const char *>(p.dout) + ro * ES, dor[r]);
      load_e<ES, E>(static_cast<const char *>(p.out) + ro * ES, of);
      float d = 0.0f;
#pragma unroll
      for (int e = 0; e < E; ++e) d = fmaf(dor[r][e], of[e], d);
      Dr[r] = wsum(d);
      Lr[r] = p.lse[(int64_t(u) * p.n + a + j) * G + h];
      if (lane == 0) p.dsum[(int64_t(u) * p.n + a + j) * G + h] = Dr[r];
    }
    if (lane == 0) qr[r][0] = 0.0f;
  }
  const int last = a + cnt - 1;
  const char *ksb = static_cast<const char *>(p.ks) + (int64_t(u) * p.n * D + lane * E) * ES;
  const char *vsb = static_cast<const char *>(p.vs) + (int64_t(u) * p.n * D + lane * E) * ES;
  const float *mk = p.mask + int64_t(u) * p.n;
  for (int s0 = 0; s0 <= last; s0 += kAhead) {
    float kk[kAhead][E], vv[kAhead][E], bias[kAhead];
#pragma unroll
    for (int i = 0; i < kAhead; ++i) {
      const int s = min(s0 + i, last);
      load_e<ES, E>(ksb + int64_t(s) * D * ES, kk[i]);
      load_e<ES, E>(vsb + int64_t(s) * D * ES, vv[i]);
      bias[i] = mk[s] * kLog2e;
    }
#pragma unroll
    for (int i = 0; i < kAhead; ++i) {
      const int s = s0 + i;
      if (s > last) break;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const int t = a + r / G;
        if (r / G >= cnt || s > t) continue;
        float d = 0.0f, dp = 0.0f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          d = fmaf(qr[r][e], kk[i][e], d);
          dp = fmaf(dor[r][e], vv[i][e], dp);
        }
        const float x = wsum(d) * p.scale_log2 + (s < t ? bias[i] : 0.0f);
        const float pr = fast_exp2(x - Lr[r]);
        const float ds = pr * (wsum(dp) - Dr[r]);
#pragma unroll
        for (int e = 0; e < E; ++e) dq[r][e] = fmaf(ds, kk[i][e], dq[r][e]);
      }
    }
  }
  const float sc = p.scale_log2 / kLog2e;   // 1 / sqrt(d)
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int j = r / G, h = r - j * G;
    if (j >= cnt) continue;
#pragma unroll
    for (int e = 0; e < E; ++e) dq[r][e] *= sc;
    if (lane == 0) dq[r][0] = 0.0f;   // q[0] reaches the loss through omega only (added later)
    store_e<ES, E>(static_cast<char *>(p.dq) + (row_q(p, b, a + j, g * G + h, D) + lane * E) * ES,
                   dq[r]);
  }
}

// Gradients of the states and of the mask entries: one wave per (unit, KB
// states), every query row (token >= state, all G heads) streamed.
template <int ES, int D, int G>
__global__ __launch_bounds__(kThreads) void train_dkv_kernel(TrainParams p, int nblocks) {
  constexpr int E = D / 64, KB = 4;
  const int lane = threadIdx.x & 63;
  const int wid = blockIdx.x * kWaves + (threadIdx.x >> 6);
  const int U = p.batch * p.hkv;
  const int u = wid / nblocks;
  if (u >= U) return;
  const int j0 = (wid - u * nblocks) * KB;
  const int kc = min(KB, p.n - j0);
  const int b = u / p.hkv, g = u - b * p.hkv;
  float kk[KB][E], vv[KB][E], bias[KB], dk[KB][E], dv[KB][E], dm[KB];
#pragma unroll
  for (int i = 0; i < KB; ++i) {
    const int s = j0 + min(i, kc - 1);
    const int64_t o = (int64_t(u) * p.n + s) * D + lane * E;
    load_e<ES, E>(static_cast<const char *>(p.ks) + o * ES, kk[i]);
    load_e<ES, E>(static_cast<const char *>(p.vs) + o * ES, vv[i]);
    bias[i] = p.mask[int64_t(u) * p.n + s] * kLog2e;
    dm[i] = 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) dk[i][e] = dv[i][e] = 0.0f;
  }
  for (int t = j0; t < p.n; ++t) {
    for (int h = 0; h < G; ++h) {
      const int64_t ro = row_q(p, b, t, g * G + h, D) + lane * E;
      float qf[E], df[E];
      load_e<ES, E>(static_cast<const char *>(p.q) + ro * ES, qf);
      load_e<ES, E>(static_cast<const char *>(p.dout) + ro * ES, df);
      if (lane == 0) qf[0] = 0.0f;
      const float L = p.lse[(int64_t(u) * p.n + t) * G + h];
      const float Dt = p.dsum[(int64_t(u) * p.n + t) * G + h];
#pragma unroll
      for (int i = 0; i < KB; ++i) {
        const int s = j0 + i;
        if (i >= kc || s > t) continue;
        float d = 0.0f, dp = 0.0f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          d = fmaf(qf[e], kk[i][e], d);
          dp = fmaf(df[e], vv[i][e], dp);
        }
        const float x = wsum(d) * p.scale_log2 + (s < t ? bias[i] : 0.0f);
        const float pr = fast_exp2(x - L);
        const float ds = pr * (wsum(dp) - Dt);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          dv[i][e] = fmaf(pr, df[e], dv[i][e]);
          dk[i][e] = fmaf(ds, qf[e], dk[i][e]);
        }
        if (s < t) dm[i] += ds;
      }
    }
  }
  const float sc = p.scale_log2 / kLog2e;
#pragma unroll
  for (int i = 0; i < KB; ++i) {
    if (i >= kc) break;
    const int64_t o = (int64_t(u) * p.n + j0 + i) * D + lane * E;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      p.dks[o + e] = dk[i][e] * sc;
      p.dvs[o + e] = dv[i][e];
    }
    if (lane == 0) p.dmask[int64_t(u) * p.n + j0 + i] = dm[i];
  }
}

// States -> tokens, part 1, one wave per (unit, 64 tokens), NT tokens at a
// time: token t feeds states j = t .. t + w - 1 with weight c_tj / z_j; its
// key and value gradients gather those states' gradients, and e_tj = d loss /
// d c_tj = ((k^_t - K~_j) . dK~_j + (v_t - V~_j) . dV~_j) / z_j is kept for
// part 2.  The NT tokens share their states, which are loaded in batches;
// per state, 1 / z_j and (K~_j . dK~_j + V~_j . dV~_j) are formed once, and
// a token's e values collect in one lane each (lane j - t) for a single
// store.
template <int ES, int D>
__global__ __launch_bounds__(64) void train_tokens_kernel(TrainParams p) {
  constexpr int E = D / 64, NT = 8, kB = 4;
  const int u = blockIdx.y, lane = threadIdx.x;
  const int b = u / p.hkv, g = u - b * p.hkv;
  const int t0 = blockIdx.x * 64, t1 = min(t0 + 64, p.n);
  const float *al = p.alpha + int64_t(u) * p.n;
  const float *om = p.omega + int64_t(u) * p.n;
  const float *zz = p.z + int64_t(u) * p.n;
  const int W = p.window;
  for (int tg = t0; tg < t1; tg += NT) {
    const int nt = min(NT, t1 - tg);
    float kt[NT][E], vt[NT][E], dk[NT][E], dv[NT][E], P[NT], wt[NT], ereg[NT];
#pragma unroll
    for (int i = 0; i < NT; ++i) {
      const int t = tg + min(i, nt - 1);
      const int64_t ro = row_k(p, b, t, g, D) + lane * E;
      load_e<ES, E>(static_cast<const char *>(p.k) + ro * ES, kt[i]);
      load_e<ES, E>(static_cast<const char *>(p.v) + ro * ES, vt[i]);
      if (lane == 0) kt[i][0] = 0.0f;
      wt[i] = om[t];
      P[i] = 1.0f;
      ereg[i] = 0.0f;
#pragma unroll
      for (int e = 0; e < E; ++e) dk[i][e] = dv[i][e] = 0.0f;
    }
    const int jl = min(tg + nt - 1 + W - 1, p.n - 1);   // last state any of them feeds
    for (int jb = tg; jb <= jl; jb += kB) {
      float dks[kB][E], dvs[kB][E], qs[kB], iz[kB], aj[kB];
#pragma unroll
      for (int q = 0; q < kB; ++q) {
        const int j = min(jb + q, jl);
        const int64_t so = (int64_t(u) * p.n + j) * D + lane * E;
        float ks[E], vs[E];
        load_e<ES, E>(static_cast<const char *>(p.ks) + so * ES, ks);
        load_e<ES, E>(static_cast<const char *>(p.vs) + so * ES, vs);
        qs[q] = 0.0f;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          dks[q][e] = p.dks[so + e];
          dvs[q][e] = p.dvs[so + e];
          qs[q] = fmaf(ks[e], dks[q][e], qs[q]);   // this lane's part of K~ . dK~ + V~ . dV~
          qs[q] = fmaf(vs[e], dvs[q][e], qs[q]);
        }
        iz[q] = 1.0f / zz[j];
        aj[q] = al[j];
      }
#pragma unroll
      for (int q = 0; q < kB; ++q) {
        const int j = jb + q;
        if (j > jl) break;
#pragma unroll
        for (int i = 0; i < NT; ++i) {
          const int t = tg + i;
          if (i >= nt || j < t || j > t + W - 1) continue;
          if (j > t) P[i] *= aj[q];            // prod_{r = t+1 .. j} alpha_r
          const float cz = wt[i] * P[i] * iz[q];
          float ev = -qs[q];
#pragma unroll
          for (int e = 0; e < E; ++e) {
            dk[i][e] = fmaf(cz, dks[q][e], dk[i][e]);
            dv[i][e] = fmaf(cz, dvs[q][e], dv[i][e]);
            ev = fmaf(kt[i][e], dks[q][e], ev);
            ev = fmaf(vt[i][e], dvs[q][e], ev);
          }
          ev = wsum(ev) * iz[q];
          if (lane == j - t) ereg[i] = ev;
        }
      }
    }
#pragma unroll
    for (int i = 0; i < NT; ++i) {
      if (i >= nt) break;
      const int t = tg + i;
      if (lane < min(W, p.n - t)) p.e[(int64_t(u) * p.n + t) * W + lane] = ereg[i];
      const int64_t ro = row_k(p, b, t, g, D) + lane * E;
      if (lane == 0) dk[i][0] = 0.0f;   // element 0 gets the decision gradient in part 2
      store_e<ES, E>(static_cast<char *>(p.dk) + ro * ES, dk[i]);
      store_e<ES, E>(static_cast<char *>(p.dv) + ro * ES, dv[i]);
    }
  }
}

// States -> tokens, part 1, on the matrix cores (bf16): one wave per (unit,
// 32 tokens t0 .. t0 + 31), which feed states t0 .. t0 + 30 + w (staged
// rows r = j - t0, NK 16-row k-steps).  Per matrix (keys, then values) the
// states' gradients, which the matrix-core state-gradient pass leaves as
// bf16 head and tail planes (dX~ = hi + lo to about 2^-17), are copied into
// LDS by direct transfers (value swizzle), and
//   E[t][j]  += X^_t . dX~_j      (A: token rows from global memory)
//   dX^T[dim][t] = sum_j dX~^T[dim][j] C^T[j][t],  C[t][j] = c_tj / z_j
// (A: transposed plane reads; B: the lane's weights, formed as in the vector
// pass, split into head and tail; hi.hi + hi.lo + lo.hi).  Then e_tj =
// (E[t][j] - K~_j . dK~_j - V~_j . dV~_j) / z_j over the window, the dot
// products left per state by the state-gradient pass.  The token gradients go out as
// whole rows through LDS.
// Two waves per SIMD, except for the widest windows at d = 128 (NK >= 4), whose
// E and transposed-product tiles need more than half the register file: one.
template <int D, int NK>
constexpr int tokens_mfma_waves() { return (D == 128 && NK >= 4) ? 1 : 2; }

template <int D, int NK>
__global__ __launch_bounds__(64, (tokens_mfma_waves<D, NK>())) void train_tokens_mfma_kernel(TrainParams p) {
  constexpr int RB = D * 2, CPR = D / 8, NTL = D / 32, KS = D / 16, ROWS = 16 * NK;
  constexpr int NCT = (ROWS + 31) / 32;   // 32-state column tiles of E and Q
  constexpr int PLANE = ROWS * RB;
  constexpr int NAL = (ROWS + 63) / 64;
  __shared__ __align__(16) unsigned char smem[2 * PLANE];
  __shared__ __align__(16) float s_al[ROWS], s_iz[ROWS];
  const int u = blockIdx.y, lane = threadIdx.x;
  const int col = lane & 31, hb = lane >> 5;
  const int b = u / p.hkv, g = u - b * p.hkv;
  const int t0 = blockIdx.x * 32;
  const int W = p.window, last = p.n - 1;
  const int64_t un = int64_t(u) * p.n;
  const int64_t plane_bytes = int64_t(p.batch) * p.hkv * p.n * RB;

  // What a phase reads from global memory, issued at once after the
  // weights are formed: the states' gradient planes (direct to LDS) and the
  // token rows (A of E).
  uint4 xa[KS];
  auto issue = [&](int m) {
    const char *hp = reinterpret_cast<const char *>(m == 0 ? p.dks : p.dvs);
#pragma unroll
    for (int i = 0; i < ROWS * CPR / 64; ++i) {
      const int c = i * 64 + lane;
      const int row = c / CPR, pc = c - row * CPR;
      const int64_t src = (un + min(t0 + row, last)) * RB + (pc ^ v_swizzle<CPR>(row)) * 16;
      dma16(smem + i * 1024, hp + src);
      dma16(smem + PLANE + i * 1024, hp + plane_bytes + src);
    }
    const char *xr = static_cast<const char *>(m == 0 ? p.k : p.v) +
                     row_k(p, b, min(t0 + col, last), g, D) * 2 + hb * 16;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) xa[ks] = ld16(xr + ks * 32);
  };

  // alpha_j and 1 / z_j of the staged states (through LDS, read as float4),
  // omega of this lane's token, 1 / z and X~ . dX~ of its E columns.
  float alv[NAL], zv[NAL], izc[NCT], qsc[NCT];
#pragma unroll
  for (int k = 0; k < NAL; ++k) {
    const int j = min(t0 + 64 * k + lane, last);
    alv[k] = p.alpha[un + j];
    zv[k] = p.z[un + j];
  }
#pragma unroll
  for (int c = 0; c < NCT; ++c) {
    izc[c] = p.z[un + min(t0 + 32 * c + col, last)];
    const int64_t jc = un + min(t0 + 32 * c + col, last);
    qsc[c] = p.qs[jc] + p.qs[int64_t(p.batch) * p.hkv * p.n + jc];
  }
  const int t = t0 + col;
  const float wt = p.omega[un + min(t, last)];
#pragma unroll
  for (int k = 0; k < NAL; ++k)
    if (64 * k + lane < ROWS) {
      s_al[64 * k + lane] = alv[k];
      s_iz[64 * k + lane] = 1.0f / zv[k];
    }
#pragma unroll
  for (int c = 0; c < NCT; ++c) izc[c] = 1.0f / izc[c];
  wave_lds_sync();

  // Weights C[t][t0 + r] of this lane's token, ascending in j as in the
  // vector pass: (omega_t prod_{r=t+1..j} alpha_r) / z_j.
  uint4 chi[NK], clo[NK];
  {
    float cw[ROWS];
    float P = 1.0f;
#pragma unroll
    for (int r4 = 0; r4 < ROWS; r4 += 4) {
      const float4 a4 = *reinterpret_cast<const float4 *>(s_al + r4);
      const float4 z4 = *reinterpret_cast<const float4 *>(s_iz + r4);
      const float av[4] = {a4.x, a4.y, a4.z, a4.w}, iv[4] = {z4.x, z4.y, z4.z, z4.w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int j = t0 + r4 + q;
        const bool in = j >= t && j < t + W && j <= last;
        if (in && j > t) P *= av[q];
        cw[r4 + q] = in ? wt * P * iv[q] : 0.0f;
      }
    }
#pragma unroll
    for (int ks = 0; ks < NK; ++ks) {
      uint32_t h[4], l[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float w0 = hb ? cw[16 * ks + 8 + 2 * q] : cw[16 * ks + 2 * q];
        const float w1 = hb ? cw[16 * ks + 9 + 2 * q] : cw[16 * ks + 1 + 2 * q];
        h[q] = cvt_pk_bf16(w0, w1);
        l[q] = cvt_pk_bf16(w0 - __uint_as_float(h[q] << 16), w1 - __uint_as_float(h[q] & 0xffff0000u));
      }
      chi[ks] = make_uint4(h[0], h[1], h[2], h[3]);
      clo[ks] = make_uint4(l[0], l[1], l[2], l[3]);
    }
  }

  uint32_t vaddr[NTL];
  {
    const int g16 = lane >> 4, r16 = lane & 15;
    const int row0 = 8 * (g16 >> 1) + (r16 >> 2);
#pragma unroll
    for (int i = 0; i < NTL; ++i) {
      const int lc = 4 * i + 2 * (g16 & 1) + ((r16 & 3) >> 1);
      vaddr[i] = row0 * RB + ((lc ^ v_swizzle<CPR>(row0)) * 16) + (r16 & 1) * 8;
    }
  }

  f32x16_t ae[NCT];
#pragma unroll
  for (int c = 0; c < NCT; ++c) ae[c] = f32x16_t{};
  const int ntok = min(32, p.n - t0);   // tokens of this block inside the sequence

#pragma unroll 1
  for (int m = 0; m < 2; ++m) {
    issue(m);
    wait_vmcnt<0>();
    wave_lds_sync();
    if (m == 0 && hb == 0) xa[0].x &= 0xffff0000u;   // k^_t: element 0 is not part of a key

    // E.
#pragma unroll
    for (int c = 0; c < NCT; ++c) {
      const int srow = 32 * c + col;
      const bool sok = srow < ROWS;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        uint4 bh = make_uint4(0, 0, 0, 0), bl = bh;
        if (sok) {
          const uint32_t off = srow * RB + (((2 * ks + hb) ^ v_swizzle<CPR>(srow)) * 16);
          bh = *reinterpret_cast<const uint4 *>(smem + off);
          bl = *reinterpret_cast<const uint4 *>(smem + PLANE + off);
        }
        ae[c] = mfma_32x32x16(xa[ks], bh, ae[c]);
        ae[c] = mfma_32x32x16(xa[ks], bl, ae[c]);
      }
    }

    // Token gradients: lane holds dims 32 i + 8 q + 4 hb .. + 4 of token t0 + col.
    f32x16_t acc[NTL];
#pragma unroll
    for (int i = 0; i < NTL; ++i) {
      acc[i] = f32x16_t{};
#pragma unroll
      for (int ks = 0; ks < NK; ++ks) {
        const uint2 h0 = ds_read_tr16(smem + vaddr[i] + 16 * ks * RB);
        const uint2 h1 = ds_read_tr16(smem + vaddr[i] + (16 * ks + 4) * RB);
        const uint2 l0 = ds_read_tr16(smem + PLANE + vaddr[i] + 16 * ks * RB);
        const uint2 l1 = ds_read_tr16(smem + PLANE + vaddr[i] + (16 * ks + 4) * RB);
        const uint4 ah = make_uint4(h0.x, h0.y, h1.x, h1.y), alo = make_uint4(l0.x, l0.y, l1.x, l1.y);
        acc[i] = mfma_32x32x16(ah, chi[ks], acc[i]);
        acc[i] = mfma_32x32x16(ah, clo[ks], acc[i]);
        acc[i] = mfma_32x32x16(alo, chi[ks], acc[i]);
      }
    }
    // Rows out through the head plane (its reads are done), chunks XOR-swizzled by row.
#pragma unroll
    for (int i = 0; i < NTL; ++i)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float x0 = acc[i][4 * q];
        if (m == 0 && i == 0 && q == 0 && hb == 0) x0 = 0.0f;   // dk[0]: the decision gradient, part 2
        const uint32_t lo = cvt_pk_bf16(x0, acc[i][4 * q + 1]);
        const uint32_t hi = cvt_pk_bf16(acc[i][4 * q + 2], acc[i][4 * q + 3]);
        *reinterpret_cast<uint2 *>(smem + col * RB + (((4 * i + q) ^ k_swizzle<CPR>(col)) * 16) + hb * 8) =
            make_uint2(lo, hi);
      }
    wave_lds_sync();
    char *dst = static_cast<char *>(m == 0 ? p.dk : p.dv);
    constexpr int RPP = 64 / CPR;
#pragma unroll
    for (int r0 = 0; r0 < 32; r0 += RPP) {
      const int row = r0 + lane / CPR, ch = lane % CPR;
      if (row < ntok)
        *reinterpret_cast<uint4 *>(dst + row_k(p, b, t0 + row, g, D) * 2 + ch * 16) =
            *reinterpret_cast<const uint4 *>(smem + row * RB + ((ch ^ k_swizzle<CPR>(row)) * 16));
    }
    wave_lds_sync();   // the planes are restaged next
  }

  // e_tj = (E[t][j] - X~_j . dX~_j) / z_j; register r of a tile is row
  // (token) t0 + 8 (r / 4) + 4 hb + r % 4, column (state) t0 + 32 c + col.
#pragma unroll
  for (int c = 0; c < NCT; ++c) {
    const int j = t0 + 32 * c + col;
    const float dq = qsc[c];
    if (j > last) continue;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int tt = t0 + 8 * (r >> 2) + 4 * hb + (r & 3);
      const int dl = j - tt;
      if (dl >= 0 && dl < W && tt <= last) p.e[(un + tt) * W + dl] = (ae[c][r] - dq) * izc[c];
    }
  }
}

// States -> tokens, part 2, one thread per (unit, token r): the weight
// gradients e give d omega_r = sum_j e_rj prod_{r+1..j} alpha and
// d alpha_r = sum_j prod_{r+1..j} alpha * sum_{t = a_j .. r-1} e_tj omega_t
// prod_{t+1..r-1} alpha; with the mask entry log(1 - alpha_r) of state r - 1
// and the caller's dalpha they reach the logit x_r, hence k_r[0] (/ tau), and
// omega reaches q_r[lead][0].
template <int ES, int D>
__global__ __launch_bounds__(kThreads) void train_neurons_kernel(TrainParams p) {
  const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  const int U = p.batch * p.hkv;
  if (i >= int64_t(U) * p.n) return;
  const int u = static_cast<int>(i / p.n), r = static_cast<int>(i - int64_t(u) * p.n);
  const int b = u / p.hkv, g = u - b * p.hkv, G = p.hq / p.hkv, W = p.window;
  const float *al = p.alpha + int64_t(u) * p.n;
  const float *om = p.omega + int64_t(u) * p.n;
  const float *ee = p.e + int64_t(u) * p.n * W;
  float domega = 0.0f, dalpha = 0.0f, S = 1.0f;
  const int jl = min(r + W - 1, p.n - 1);
  for (int j = r; j <= jl; ++j) {
    if (j > r) S *= al[j];                   // prod_{r' = r+1 .. j} alpha
    domega = fmaf(ee[int64_t(r) * W + (j - r)], S, domega);
    const int aj = max(0, j - W + 1);
    if (aj < r) {
      float F = 0.0f, Q = 1.0f;
      for (int t = r - 1; t >= aj; --t) {     // Q = prod_{t+1 .. r-1} alpha
        F = fmaf(ee[int64_t(t) * W + (j - t)] * om[t], Q, F);
        Q *= al[t];
      }
      dalpha = fmaf(S, F, dalpha);
    }
  }
  const float a_r = al[r];
  if (p.dalpha) dalpha += p.dalpha[(int64_t(b) * p.n + r) * p.hkv + g];
  float dx = dalpha * a_r * (1.0f - a_r);
  if (r > 0) dx -= a_r * p.dmask[int64_t(u) * p.n + r - 1];   // d log(1 - sigmoid(x)) / dx = -alpha
  float dk0 = dx / p.tau;
  if constexpr (ES == 2) {
    static_cast<uint16_t *>(p.dk)[row_k(p, b, r, g, D)] = static_cast<uint16_t>(bf16_bits(dk0));
  } else {
    static_cast<float *>(p.dk)[row_k(p, b, r, g, D)] = dk0;
  }
  if (p.omega_src == 0) {
    const float w = om[r];
    const float dq0 = w > 0x1p-100f ? domega * w * (1.0f - w) : 0.0f;
    if constexpr (ES == 2) {
      static_cast<uint16_t *>(p.dq)[row_q(p, b, r, g * G, D)] = static_cast<uint16_t>(bf16_bits(dq0));
    } else {
      static_cast<float *>(p.dq)[row_q(p, b, r, g * G, D)] = dq0;
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 attention on the matrix cores.
//
// Query-major kernels (forward, dq): one workgroup = 4 waves = 128 query
// columns of one unit, token-major (column c = token c / G, head c % G); a
// wave owns 32 columns.  The unit's states stream through LDS in blocks of 32
// rows (direct global -> LDS transfers, a 4-slot ring three blocks ahead), and
// per block and wave, lane l holding column l % 32 and half l / 32:
//   S^T[state][col] = K'[state] . Q'[col]     (A = K' rows, B = Q'^T)
// Score row m is state pi(m) (bits 2 and 3 of m swapped), so a lane's score
// registers 8 kk .. 8 kk + 7 are its B-operand slice for states
// 16 kk + 8 half .. + 8 of the products that contract over states:
//   forward: O^T[dim][col] += V^T[dim][state] P^T[state][col]
//   dq:      dQ^T[dim][col] += K^T[dim][state] dS^T[state][col]
// The mask is folded into the score product: key-state element 0 holds the
// state's mask entry times sqrt(d) and query element 0 is set to 1 (neither
// is otherwise part of a score); the diagonal takes it out again, and states
// past a column's token are masked in the blocks that reach the diagonal.
//
// State-major kernel (dK~, dV~, mask gradient): one workgroup = 4 waves =
// 128 states of one unit, a wave owning 32 (its K~, V~ rows are operands in
// registers); query rows (token, head) stream through LDS in blocks of 32
// (a 3-slot ring):
//   S[row][state] = Q[row] . K~[state],  dP[row][state] = dO[row] . V~[state]
// with rows pi-permuted so that P^T and dS^T come out as A operands of
//   dV~[state][dim] += P^T[state][row] dO[row][dim]
//   dK~[state][dim] += dS^T[state][row] Q[row][dim].
// Rows read as "8 consecutive rows of one dim" (V^T, K^T, dO, Q) use the
// transposed LDS read ds_read_b64_tr_b16 on rows stored with the value
// swizzle.
// ---------------------------------------------------------------------------

// Ring slots (blocks in flight + 1) of the query-major kernels (64 KiB of
// LDS per workgroup, two per CU) and of the state-major ones (three per CU
// at 3 slots; 4 slots measured slower there, faster for forward and dq).
constexpr int kQMajorStages = 4, kDkvStages = 3;

// Waits until the ring block of step kb has landed: `after` blocks were
// issued behind it, PER transfers each.
template <int PER>
__device__ __forceinline__ void wait_block(int after) {
  if (after >= 2) wait_vmcnt<2 * PER>();
  else if (after == 1) wait_vmcnt<PER>();
  else wait_vmcnt<0>();
}

// Swizzle of a block's rows: 0 key (row reads), 1 value (transposed reads),
// 2 dual (both).
template <int CPR, int SW>
__device__ __forceinline__ int block_swizzle(int row) {
  return SW == 0 ? k_swizzle<CPR>(row) : SW == 1 ? v_swizzle<CPR>(row) : dual_swizzle<CPR>(row);
}

// Transposed operand: A or B slice "rows 16 kk + 8 half + 0..7 of dim 32 t +
// col" of a 32-row block (vaddr[t][h]: offsets of the two 4-row halves).
template <int RB>
__device__ __forceinline__ uint4 tr_operand(const char *blk, const uint32_t (&vaddr)[2], int kk) {
  const uint2 h0 = ds_read_tr16(blk + vaddr[0] + 16 * kk * RB);
  const uint2 h1 = ds_read_tr16(blk + vaddr[1] + 16 * kk * RB);
  return make_uint4(h0.x, h0.y, h1.x, h1.y);
}

// Per-lane offsets of the transposed reads (per 32-dim tile and 4-row half)
// for a block stored with swizzle SW (1 or 2): a 16-lane group points at
// four 8-byte pieces of each of 4 rows.
template <int D, int SW>
__device__ __forceinline__ void tr_offsets(int lane, uint32_t (&vaddr)[D / 32][2]) {
  constexpr int RB = D * 2, CPR = D / 8;
  const int g16 = lane >> 4, r16 = lane & 15;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int row = 8 * (g16 >> 1) + 4 * h + (r16 >> 2);
#pragma unroll
    for (int t = 0; t < D / 32; ++t) {
      const int lc = 4 * t + 2 * (g16 & 1) + ((r16 & 3) >> 1);
      vaddr[t][h] = row * RB + ((lc ^ block_swizzle<CPR, SW>(row)) * 16) + (r16 & 1) * 8;
    }
  }
}

// Row-read offsets: 16 bytes (dims 16 ks + 8 half .. + 8) of row `row` of a
// block stored with swizzle SW.
template <int D, int SW>
__device__ __forceinline__ uint32_t row_offset(int row, int ks, int hb) {
  constexpr int RB = D * 2, CPR = D / 8;
  return row * RB + (((2 * ks + hb) ^ block_swizzle<CPR, SW>(row)) * 16);
}

// Query-major kernels: MODE 0 = forward, 1 = dq.
template <int D, int G, int MODE>
__global__ __launch_bounds__(kThreads, 2) void train_qmajor_kernel(TrainParams p, int ntiles) {
  constexpr int kSt = kQMajorStages;   // ring slots
  constexpr int T = 32 / G;            // tokens per wave
  constexpr int TW = kWaves * T;       // tokens per workgroup
  constexpr int KS = D / 16;           // 16-dim k-steps of the score product
  constexpr int NTL = D / 32;          // 32-dim tiles of the contraction over states
  constexpr int RB = D * 2;
  constexpr int CPR = D / 8;
  constexpr int BLK = 32 * RB;
  constexpr int DPW = BLK / 16 / kThreads;
  constexpr int KSW = MODE == 0 ? 0 : 2;   // dq also reads keys transposed
  constexpr int VSW = MODE == 0 ? 1 : KSW;   // forward reads values transposed; dq as rows,
                                             // laid out like the keys (shared offsets)
  static_assert(DPW >= 1 && BLK % (16 * kThreads) == 0, "block split");
  static_assert(kSt == 4, "the block loop below is unrolled for four slots");
  // The state ring, one array per slot (see dma16_s): keys, then values.
  __shared__ __align__(16) unsigned char ring0[2 * BLK], ring1[2 * BLK], ring2[2 * BLK],
      ring3[2 * BLK];
  auto slot = [&](auto st_c) -> unsigned char * {
    constexpr int S = decltype(st_c)::value;
    if constexpr (S == 0) return ring0;
    else if constexpr (S == 1) return ring1;
    else if constexpr (S == 2) return ring2;
    else return ring3;
  };

  const int U = p.batch * p.hkv;
  const int bid = blockIdx.x;
  const int xcd = bid & 7, r = bid >> 3;
  const int ul = r / ntiles, tile = ntiles - 1 - (r - ul * ntiles);
  const int u = ul * 8 + xcd;
  if (u >= U) return;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, hb = lane >> 5;
  const int b = u / p.hkv, g = u - b * p.hkv;
  const int a = tile * TW + wave * T;
  const int cnt = max(0, min(T, p.n - a));
  const int tok = col / G, head = col - tok * G;
  const bool colv = tok < cnt;
  const int t = a + tok;
  const uint4 zero4 = make_uint4(0, 0, 0, 0);
  const int s_top = min(p.n, tile * TW + TW);   // states 0 .. s_top - 1 feed this tile
  const int nblk = (s_top + 31) >> 5;
  const int wave_hi = a + cnt;                  // states < wave_hi feed this wave
  const float sl2 = p.scale_log2;

  // Q'^T operand: Q[col][16 ks + 8 hb .. + 8] with element 0 set to 1.
  uint4 qop[KS], dop[MODE == 1 ? KS : 1];
  float Lc = 0.0f, Dc = 0.0f, diag = 0.0f;
  {
    const int64_t ro = row_q(p, b, colv ? t : 0, g * G + head, D);
    const char *qr = static_cast<const char *>(p.q) + ro * 2;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qop[ks] = colv ? ld16(qr + ks * 32 + hb * 16) : zero4;
    if (hb == 0) qop[0].x = (qop[0].x & 0xffff0000u) | 0x3f80u;
    // the diagonal state's mask entry as stored (bf16 of mask * sqrt(d))
    if (colv) {
      const float md = p.mask[int64_t(u) * p.n + t] * (kLog2e / sl2);
      diag = __uint_as_float(bf16_bits(md) << 16);
    }
    if constexpr (MODE == 1) {
      const char *dr = static_cast<const char *>(p.dout) + ro * 2;
      const char *orow = static_cast<const char *>(p.out) + ro * 2;
      float part = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        dop[ks] = colv ? ld16(dr + ks * 32 + hb * 16) : zero4;
        const uint4 ov = colv ? ld16(orow + ks * 32 + hb * 16) : zero4;
        float df[8], of[8];
        V16<2>::unpack(dop[ks], df);
        V16<2>::unpack(ov, of);
#pragma unroll
        for (int e = 0; e < 8; ++e) part = fmaf(df[e], of[e], part);
      }
      Dc = part + __shfl_xor(part, 32, 64);
      if (colv) Lc = p.lse[(int64_t(u) * p.n + t) * G + head];
      if (colv && hb == 0) p.dsum[(int64_t(u) * p.n + t) * G + head] = Dc;
    }
  }

  float m = -1e30f, ls = 0.0f;
  f32x16_t acc[NTL];
#pragma unroll
  for (int i = 0; i < NTL; ++i) acc[i] = f32x16_t{};

  // Block transfers (same chunk mapping as prompt attention; the unit's
  // states are contiguous, so one wave-uniform base per block).  Every call
  // issues 2 DPW transfers per wave; those of blocks past the last one are
  // switched off.
  uint32_t koff[DPW], voff[MODE == 0 ? DPW : 1];
#pragma unroll
  for (int i = 0; i < DPW; ++i) {
    const int c = (i * kWaves + wave) * 64 + lane;
    const int row = c / CPR, pc = c - row * CPR;
    koff[i] = row * RB + (pc ^ block_swizzle<CPR, KSW>(row)) * 16;
    if constexpr (MODE == 0) voff[i] = row * RB + (pc ^ block_swizzle<CPR, VSW>(row)) * 16;
  }
  const char *kst = static_cast<const char *>(p.ks) + int64_t(u) * p.n * RB;
  const char *vst = static_cast<const char *>(p.vs) + int64_t(u) * p.n * RB;
  auto issue = [&](int kb, auto st_c) {
    const bool on = kb < nblk;
#pragma unroll
    for (int i = 0; i < DPW; ++i) {
      unsigned char *kdst = slot(st_c) + (i * kWaves + wave) * 1024;
      dma16_s(kdst, uniform_ptr(kst + int64_t(kb) * BLK), koff[i], on);
      dma16_s(kdst + BLK, uniform_ptr(vst + int64_t(kb) * BLK), MODE == 0 ? voff[i] : koff[i], on);
    }
  };

  const int krow = score_slot(col);
  uint32_t kaddr[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    kaddr[ks] = row_offset<D, KSW>(krow, ks, hb);
  }
  uint32_t traddr[NTL][2];
  tr_offsets<D, MODE == 0 ? VSW : KSW>(lane, traddr);

  // One block of the dq kernel.
  auto step = [&](auto stage_c, int kb) {
    constexpr int ST = decltype(stage_c)::value;
    wait_vmcnt<(kSt - 2) * 2 * DPW>();   // block kb has landed
    ring_barrier();   // block kb is in LDS for every wave; the slot of kb - 1 is free
    issue(kb + kSt - 1, std::integral_constant<int, (ST + kSt - 1) % kSt>{});
    if (kb * 32 >= wave_hi) return;
    const char *kd = reinterpret_cast<const char *>(slot(stage_c));
    const char *vd = kd + BLK;

    f32x16_t sc = f32x16_t{};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      sc = mfma_32x32x16(*reinterpret_cast<const uint4 *>(kd + kaddr[ks]), qop[ks], sc);
    float sv[16];
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) sv[rr] = sc[rr];
    if (kb * 32 + 32 > a) {   // the block reaches the diagonal
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const int st = kb * 32 + score_slot(8 * (rr >> 2) + 4 * hb + (rr & 3));
        if (st > t) sv[rr] = neg_inf();
        else if (st == t) sv[rr] -= diag;
      }
    }
    {   // dq (the forward runs the pipelined step below)
      // dP^T = V . dO^T, with P = exp2(S - L) (the forward's statistics)
      // formed between its MFMAs (order pinned; value rows read two ahead),
      // then dS^T = P^T (dP^T - D).
      f32x16_t dp = f32x16_t{};
      float pe[16];
      uint4 vr[3];
      vr[0] = *reinterpret_cast<const uint4 *>(vd + kaddr[0]);
      vr[1] = *reinterpret_cast<const uint4 *>(vd + kaddr[1]);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if (ks + 2 < KS) vr[(ks + 2) % 3] = *reinterpret_cast<const uint4 *>(vd + kaddr[ks + 2]);
        dp = mfma_32x32x16(vr[ks % 3], dop[ks], dp);
#pragma unroll
        for (int e = 0; e < 16 / KS; ++e) {
          const int i = ks * (16 / KS) + e;
          pe[i] = fast_exp2(fmaf(sv[i], sl2, -Lc));
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      uint4 sb[2];
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        uint32_t w[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int r0 = 8 * kk + 2 * q;
          w[q] = cvt_pk_bf16(pe[r0] * (dp[r0] - Dc), pe[r0 + 1] * (dp[r0 + 1] - Dc));
        }
        sb[kk] = make_uint4(w[0], w[1], w[2], w[3]);
      }
#pragma unroll
      for (int i = 0; i < NTL; ++i)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
          acc[i] = mfma_32x32x16(tr_operand<RB>(kd, traddr[i], kk), sb[kk], acc[i]);
    }
  };

  issue(0, std::integral_constant<int, 0>{});
  issue(1, std::integral_constant<int, 1>{});
  issue(2, std::integral_constant<int, 2>{});
  if constexpr (MODE == 0) {
    // Step kb runs block kb's exponentials between the score MFMAs of block
    // kb + 1 (one accumulator chain; order pinned by scheduling barriers),
    // then block kb's value product.
    f32x16_t scn = f32x16_t{};
    if (nblk > 0) {
      wait_vmcnt<(kSt - 2) * 2 * DPW>();   // block 0 has landed
      ring_barrier();
      if (wave_hi > 0) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          scn = mfma_32x32x16(*reinterpret_cast<const uint4 *>(
                                  reinterpret_cast<const char *>(ring0) + kaddr[ks]), qop[ks], scn);
      }
    }
    auto step0 = [&](auto stage_c, int kb) {
      constexpr int ST = decltype(stage_c)::value, SN = (ST + 1) % kSt;
      wait_vmcnt<(kSt - 3) * 2 * DPW>();   // block kb + 1 has landed
      ring_barrier();   // every wave is past step kb - 1: the slot of kb - 1 is free
      issue(kb + kSt - 1, std::integral_constant<int, (ST + kSt - 1) % kSt>{});
      if (kb * 32 >= wave_hi) return;
      const char *vd = reinterpret_cast<const char *>(slot(stage_c)) + BLK;
      const char *kn = reinterpret_cast<const char *>(slot(std::integral_constant<int, SN>{}));   // block kb + 1's keys
      float sv[16];
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) sv[rr] = scn[rr];
      if (kb * 32 + 32 > a) {   // the block reaches the diagonal
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int st = kb * 32 + score_slot(8 * (rr >> 2) + 4 * hb + (rr & 3));
          if (st > t) sv[rr] = neg_inf();
          else if (st == t) sv[rr] -= diag;
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
        for (int i = 0; i < NTL; ++i) acc[i] *= f;
      }
      // The next block's slot always holds readable data; past the last
      // block its scores are not used.
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
#pragma unroll
      for (int i = 0; i < NTL; ++i)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
          acc[i] = mfma_32x32x16(tr_operand<RB>(vd, traddr[i], kk), pb[kk], acc[i]);
    };
    // Whole rounds of four steps (a step past the last block only keeps the
    // barriers and transfer counts in step).
    for (int kb = 0; kb < nblk; kb += kSt) {
      step0(std::integral_constant<int, 0>{}, kb);
      step0(std::integral_constant<int, 1>{}, kb + 1);
      step0(std::integral_constant<int, 2>{}, kb + 2);
      step0(std::integral_constant<int, 3>{}, kb + 3);
    }
  } else {
    for (int kb = 0; kb < nblk; kb += kSt) {
      step(std::integral_constant<int, 0>{}, kb);
      step(std::integral_constant<int, 1>{}, kb + 1);
      step(std::integral_constant<int, 2>{}, kb + 2);
      step(std::integral_constant<int, 3>{}, kb + 3);
    }
  }

  // Lane holds dims 32 i + 8 j + 4 hb .. + 4 of its column.
  if (!colv) return;
  char *orow = static_cast<char *>(MODE == 0 ? p.out : p.dq) + row_q(p, b, t, g * G + head, D) * 2;
  float sc_out;
  if constexpr (MODE == 0) {
    const float lt = ls + __shfl_xor(ls, 32, 64);
    sc_out = 1.0f / lt;
    if (hb == 0) p.lse[(int64_t(u) * p.n + t) * G + head] = m + __log2f(lt);
  } else {
    sc_out = sl2 / kLog2e;   // 1 / sqrt(d)
  }
#pragma unroll
  for (int i = 0; i < NTL; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float x0 = acc[i][4 * j] * sc_out, x1 = acc[i][4 * j + 1] * sc_out;
      if (MODE == 1 && i == 0 && j == 0 && hb == 0) x0 = 0.0f;   // dq[0]: through omega only
      const uint32_t lo = cvt_pk_bf16(x0, x1);
      const uint32_t hi = cvt_pk_bf16(acc[i][4 * j + 2] * sc_out, acc[i][4 * j + 3] * sc_out);
      *reinterpret_cast<uint2 *>(orow + (32 * i + 8 * j + 4 * hb) * 2) = make_uint2(lo, hi);
    }
}

// State-major kernel: dK~, dV~ and the mask gradient of 128 states per
// workgroup (32 per wave); query rows (token-major, G per token) stream
// through LDS in blocks of 32 rows.  PART 1 computes dV~ (S, P), PART 2 dK~
// and the mask gradient (S, dP, dS): each holds half the accumulators of a
// combined kernel and runs at least two waves per SIMD (measured about 10 %
// faster together than the combined kernel at one wave per SIMD).
template <int D, int G, int PART>
__global__ __launch_bounds__(kThreads, 2) void train_dkv_mfma_kernel(TrainParams p, int ntiles) {
  static_assert(PART == 1 || PART == 2, "dV part or dK part");
  constexpr int kSt = kDkvStages;
  constexpr int KS = D / 16, NTL = D / 32, RB = D * 2, CPR = D / 8, BLK = 32 * RB;
  constexpr int DPW = BLK / 16 / kThreads;
  // One ring slot: query rows, dO rows, then per wave its own copy of the
  // block's statistics (32 L, then 32 D).  Three workgroups (3 x 52 KB at
  // d = 128) share a compute unit.
  constexpr int SLOT = 2 * BLK + kWaves * 256;
  static_assert(DPW >= 1, "block split");
  static_assert(kSt == 3, "the block loop below is unrolled for three slots");
  __shared__ __align__(16) unsigned char ring0[SLOT], ring1[SLOT], ring2[SLOT];
  auto slot = [&](auto st_c) -> unsigned char * {
    constexpr int S = decltype(st_c)::value;
    if constexpr (S == 0) return ring0;
    else if constexpr (S == 1) return ring1;
    else return ring2;
  };

  const int U = p.batch * p.hkv;
  const int bid = blockIdx.x;
  const int xcd = bid & 7, r = bid >> 3;
  const int ul = r / ntiles, tile = r - ul * ntiles;   // earliest states (most rows) first
  const int u = ul * 8 + xcd;
  if (u >= U) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 31, hb = lane >> 5;
  const int b = u / p.hkv, g = u - b * p.hkv;
  const int s0 = tile * 128 + wave * 32;             // this wave's first state
  const int js = s0 + col;                            // this lane's state (column)
  const bool sv_ok = js < p.n;
  const uint4 zero4 = make_uint4(0, 0, 0, 0);
  const float sl2 = p.scale_log2;

  // K~ and V~ of the lane's state as B operands (dims 16 ks + 8 hb .. + 8).
  // Key element 0 carries the state's mask entry (bf16 of mask * sqrt(d));
  // the query operand's element 0 is set to 1, so every score arrives with
  // the bias of a past row, which the diagonal takes out again.
  uint4 kop[KS], vop[KS];
  float bias = 0.0f;
  {
    const int64_t so = (int64_t(u) * p.n + (sv_ok ? js : 0)) * RB;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      kop[ks] = sv_ok ? ld16(static_cast<const char *>(p.ks) + so + ks * 32 + hb * 16) : zero4;
      vop[ks] = (sv_ok && PART != 1) ? ld16(static_cast<const char *>(p.vs) + so + ks * 32 + hb * 16)
                                     : zero4;
    }
    // the same entry in log2 units
    if (sv_ok)
      bias = __uint_as_float(bf16_bits(p.mask[int64_t(u) * p.n + js] * (kLog2e / sl2)) << 16) * sl2;
  }

  // Query rows r = t * G + h; the workgroup needs rows of tokens >= its
  // first state.
  const int row_lo = tile * 128 * G;
  const int nrows = p.n * G;
  const int qb0 = row_lo >> 5, qb1 = (nrows + 31) >> 5;
  const int nblk = qb1 - qb0;
  // This thread's chunks: block row loff, byte offset qoff within the row (a
  // block's rows r = t G + h are 32 / G whole tokens).
  uint32_t qoff[DPW], loff[DPW];
#pragma unroll
  for (int i = 0; i < DPW; ++i) {
    const int c = (i * kWaves + wave) * 64 + lane;
    const int row = c / CPR, pc = c - row * CPR;
    loff[i] = row;
    qoff[i] = (pc ^ dual_swizzle<CPR>(row)) * 16;
  }
  const int64_t row0 = row_q(p, b, 0, g * G, D) * 2;   // bytes to (b, token 0, head g G)
  const int64_t tokb = int64_t(p.hq) * D * 2;          // bytes per token
  // Every call issues 2 DPW + 1 transfers per wave; those of blocks past the
  // last one are switched off.  Rows past the sequence (the last block) read
  // its last row: in bounds and finite, masked when used.  Each wave copies
  // the block's statistics ([U][n][G] rows, padded by 32) into its own area
  // by one 4-byte transfer: lanes 0..31 L of the 32 rows, lanes 32..63 their
  // D, which lies a fixed distance after L in the workspace (under 2^28
  // bytes: the API limits the query tensor to 2^31 elements).
  const char *lse_u = reinterpret_cast<const char *>(p.lse) + int64_t(u) * p.n * G * 4;
  const uint32_t dsum_delta = static_cast<uint32_t>(reinterpret_cast<const char *>(p.dsum) -
                                                    reinterpret_cast<const char *>(p.lse));
  const uint32_t soff_lane = uint32_t(lane & 31) * 4 + (lane >= 32 ? dsum_delta : 0u);
  auto issue = [&](int qb, auto st_c) {
    const bool on = qb < qb1;
    unsigned char *dst = slot(st_c);
    const int64_t bb = row0 + int64_t(qb * (32 / G)) * tokb;
    const char *qp = uniform_ptr(static_cast<const char *>(p.q) + bb);
    const char *dp = uniform_ptr(static_cast<const char *>(p.dout) + bb);
    const int last_rel = nrows - 1 - qb * 32;   // the block's last row inside the sequence
#pragma unroll
    for (int i = 0; i < DPW; ++i) {
      unsigned char *cdst = dst + (i * kWaves + wave) * 1024;
      const int rel = min(int(loff[i]), last_rel);
      const uint32_t off = uint32_t(((rel / G) * p.hq + rel % G) * D * 2) + qoff[i];
      dma16_s(cdst, qp, off, on);
      dma16_s(cdst + BLK, dp, off, on);
    }
    dma_so<kCachePolicyDefault, 4>(dst + 2 * BLK + wave * 256, uniform_ptr(lse_u),
                                   soff_lane + uint32_t(qb) * 128, on);
  };
  const int qrow = score_slot(col);
  uint32_t raddr[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) raddr[ks] = row_offset<D, 2>(qrow, ks, hb);
  uint32_t traddr[NTL][2];
  tr_offsets<D, 2>(lane, traddr);

  f32x16_t dk[NTL], dv[NTL];
#pragma unroll
  for (int i = 0; i < NTL; ++i) dk[i] = dv[i] = f32x16_t{};
  float dm = 0.0f;

  auto step = [&](auto stage_c, int kb) {
    constexpr int ST = decltype(stage_c)::value;
    wait_vmcnt<(kSt - 2) * (2 * DPW + 1)>();   // block kb has landed
    ring_barrier();   // block kb is in LDS for every wave; the slot of kb - 1 is free
    issue(qb0 + kb + kSt - 1, std::integral_constant<int, (ST + kSt - 1) % kSt>{});
    const int rb = (qb0 + kb) * 32;                  // first row of the block
    if (kb >= nblk || rb + 31 < s0 * G) return;      // past the last block, or every row
                                                     // precedes this wave's states
    const char *qd = reinterpret_cast<const char *>(slot(stage_c));
    const char *dd = qd + BLK;
    const bool interior = rb / G > s0 + 31 && rb + 32 <= nrows && s0 + 32 <= p.n;
    f32x16_t sc = f32x16_t{}, dp = f32x16_t{};
    // Softmax statistics of register 8 kk + q of this lane: row rb + 16 kk +
    // 8 hb + q (pi-permuted rows), from this wave's copy of the block's
    // statistics (L rows at sl, D rows at sl + 32).
    const float *sl = reinterpret_cast<const float *>(qd + 2 * BLK + wave * 256);
    uint4 pa[2], da[2];
    if (PART == 2 && interior) {
      // Scores first; then dP's MFMAs with P's exponentials between them
      // (order pinned; dO rows read two ahead).
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        uint4 qa = *reinterpret_cast<const uint4 *>(qd + raddr[ks]);
        if (ks == 0 && hb == 0) qa.x = (qa.x & 0xffff0000u) | 0x3f80u;   // query element 0 <- 1
        sc = mfma_32x32x16(qa, kop[ks], sc);
      }
      float Lr[16], Dr[16];
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const float *e8 = sl + 16 * kk + 8 * hb;
#pragma unroll
        for (int c4 = 0; c4 < 2; ++c4) {
          const float4 l4 = *reinterpret_cast<const float4 *>(e8 + 4 * c4);
          const float4 d4 = *reinterpret_cast<const float4 *>(e8 + 32 + 4 * c4);
          Lr[8 * kk + 4 * c4 + 0] = l4.x; Lr[8 * kk + 4 * c4 + 1] = l4.y;
          Lr[8 * kk + 4 * c4 + 2] = l4.z; Lr[8 * kk + 4 * c4 + 3] = l4.w;
          Dr[8 * kk + 4 * c4 + 0] = d4.x; Dr[8 * kk + 4 * c4 + 1] = d4.y;
          Dr[8 * kk + 4 * c4 + 2] = d4.z; Dr[8 * kk + 4 * c4 + 3] = d4.w;
        }
      }
      float pe[16];
      uint4 dr[3];
      dr[0] = *reinterpret_cast<const uint4 *>(dd + raddr[0]);
      dr[1] = *reinterpret_cast<const uint4 *>(dd + raddr[1]);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        if (ks + 2 < KS) dr[(ks + 2) % 3] = *reinterpret_cast<const uint4 *>(dd + raddr[ks + 2]);
        dp = mfma_32x32x16(dr[ks % 3], vop[ks], dp);
#pragma unroll
        for (int e = 0; e < 16 / KS; ++e) {
          const int i = ks * (16 / KS) + e;
          pe[i] = fast_exp2(fmaf(sc[i], sl2, -Lr[i]));
        }
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        uint32_t wd[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int i = 8 * kk + 2 * q;
          const float d0 = pe[i] * (dp[i] - Dr[i]), d1 = pe[i + 1] * (dp[i + 1] - Dr[i + 1]);
          dm += d0;
          dm += d1;
          wd[q] = cvt_pk_bf16(d0, d1);
        }
        da[kk] = make_uint4(wd[0], wd[1], wd[2], wd[3]);
        pa[kk] = da[kk];   // unused by this part
      }
    } else {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      uint4 qa = *reinterpret_cast<const uint4 *>(qd + raddr[ks]);
      if (ks == 0 && hb == 0) qa.x = (qa.x & 0xffff0000u) | 0x3f80u;   // query element 0 <- 1
      sc = mfma_32x32x16(qa, kop[ks], sc);
      if constexpr (PART != 1)
        dp = mfma_32x32x16(*reinterpret_cast<const uint4 *>(dd + raddr[ks]), vop[ks], dp);
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      float Lr[16], Dr[16];   // indexed by register 8 kk + q: only this kk's half is loaded
      {
        const float *e8 = sl + 16 * kk + 8 * hb;
        const float4 l0 = *reinterpret_cast<const float4 *>(e8);
        const float4 l1 = *reinterpret_cast<const float4 *>(e8 + 4);
        Lr[8 * kk + 0] = l0.x; Lr[8 * kk + 1] = l0.y; Lr[8 * kk + 2] = l0.z; Lr[8 * kk + 3] = l0.w;
        Lr[8 * kk + 4] = l1.x; Lr[8 * kk + 5] = l1.y; Lr[8 * kk + 6] = l1.z; Lr[8 * kk + 7] = l1.w;
        if constexpr (PART != 1) {
          const float4 d0 = *reinterpret_cast<const float4 *>(e8 + 32);
          const float4 d1 = *reinterpret_cast<const float4 *>(e8 + 36);
          Dr[8 * kk + 0] = d0.x; Dr[8 * kk + 1] = d0.y; Dr[8 * kk + 2] = d0.z; Dr[8 * kk + 3] = d0.w;
          Dr[8 * kk + 4] = d1.x; Dr[8 * kk + 5] = d1.y; Dr[8 * kk + 6] = d1.z; Dr[8 * kk + 7] = d1.w;
        } else {
#pragma unroll
          for (int q = 0; q < 8; ++q) Dr[8 * kk + q] = 0.0f;
        }
      }
      uint32_t wp[4], wd[4];
      if (interior) {   // every row's token is past every state of the wave
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float pv[2], dsv[2];
#pragma unroll
          for (int e = 0; e < 2; ++e) {
            const int i = 8 * kk + 2 * q + e;
            pv[e] = fast_exp2(fmaf(sc[i], sl2, -Lr[i]));
            dsv[e] = pv[e] * (dp[i] - Dr[i]);
            dm += dsv[e];
          }
          wp[q] = cvt_pk_bf16(pv[0], pv[1]);
          wd[q] = cvt_pk_bf16(dsv[0], dsv[1]);
        }
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float pv[2], dsv[2];
#pragma unroll
          for (int e = 0; e < 2; ++e) {
            const int i = 8 * kk + 2 * q + e;
            const int rg = rb + 16 * kk + 8 * hb + 2 * q + e;
            const int tq = rg / G;
            const bool vis = sv_ok && rg < nrows && tq >= js;
            const float x = sc[i] * sl2 - (tq > js ? 0.0f : bias);   // no bias on the diagonal
            pv[e] = vis ? fast_exp2(x - Lr[i]) : 0.0f;
            dsv[e] = vis ? pv[e] * (dp[i] - Dr[i]) : 0.0f;   // statistics past the rows are not read
            if (vis && tq > js) dm += dsv[e];
          }
          wp[q] = cvt_pk_bf16(pv[0], pv[1]);
          wd[q] = cvt_pk_bf16(dsv[0], dsv[1]);
        }
      }
      pa[kk] = make_uint4(wp[0], wp[1], wp[2], wp[3]);
      da[kk] = make_uint4(wd[0], wd[1], wd[2], wd[3]);
    }
    }
#pragma unroll
    for (int i = 0; i < NTL; ++i)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        if constexpr (PART != 2) dv[i] = mfma_32x32x16(pa[kk], tr_operand<RB>(dd, traddr[i], kk), dv[i]);
        if constexpr (PART != 1) dk[i] = mfma_32x32x16(da[kk], tr_operand<RB>(qd, traddr[i], kk), dk[i]);
      }
  };

  issue(qb0, std::integral_constant<int, 0>{});
  issue(qb0 + 1, std::integral_constant<int, 1>{});
  // Whole rounds of three steps (a step past the last block only keeps the
  // barriers and transfer counts in step).
  for (int kb = 0; kb < nblk; kb += kSt) {
    step(std::integral_constant<int, 0>{}, kb);
    step(std::integral_constant<int, 1>{}, kb + 1);
    step(std::integral_constant<int, 2>{}, kb + 2);
  }

  // Outputs: C[state][dim] -- lane holds dim 32 i + col of states
  // s0 + 8 (j / 4) + 4 hb + j % 4.
  if constexpr (PART != 1) {
    dm += __shfl_xor(dm, 32, 64);
    if (hb == 0 && sv_ok) p.dmask[int64_t(u) * p.n + js] = dm;
  }
  // dK~ and dV~ leave as bf16 head and tail planes ([U][n][D] each, in the
  // fp32 array's bytes): x = hi + lo to about 2^-17, the operand form the
  // token pass stages straight into LDS.  Then X~_j . dX~_j of the wave's
  // states for the token pass (value and key parts in two arrays): per
  // state, the lanes of a half hold its 32-dim slices.
  const float sc_k = sl2 / kLog2e;
  const int64_t plane = int64_t(U) * p.n * D;
  auto emit = [&](auto part_c) {
    constexpr int PT = decltype(part_c)::value;
    auto grad = [&](int i, int j) {
      const int dim = 32 * i + col;
      if constexpr (PT == 1) return dv[i][j];
      else return dim == 0 ? 0.0f : dk[i][j] * sc_k;
    };
    uint16_t *out = reinterpret_cast<uint16_t *>(PT == 1 ? p.dvs : p.dks);
#pragma unroll
    for (int i = 0; i < NTL; ++i)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int st = s0 + 8 * (j >> 2) + 4 * hb + (j & 3);
        if (st >= p.n) continue;
        const int64_t o = (int64_t(u) * p.n + st) * D + 32 * i + col;
        const float x = grad(i, j);
        const uint32_t h = bf16_bits(x);
        out[o] = static_cast<uint16_t>(h);
        out[plane + o] = static_cast<uint16_t>(bf16_bits(x - __uint_as_float(h << 16)));
      }
    const uint16_t *xs = reinterpret_cast<const uint16_t *>(PT == 1 ? p.vs : p.ks);
    float part[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int st = min(s0 + 8 * (j >> 2) + 4 * hb + (j & 3), p.n - 1);
      part[j] = 0.0f;
#pragma unroll
      for (int i = 0; i < NTL; ++i) {
        const float xv = __uint_as_float(uint32_t(xs[(int64_t(u) * p.n + st) * D + 32 * i + col]) << 16);
        part[j] = fmaf(xv, grad(i, j), part[j]);
      }
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) part[j] = row_sum<32>(part[j]);
    if (col == 0) {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int st = s0 + 8 * (j >> 2) + 4 * hb + (j & 3);
        if (st >= p.n) continue;
        p.qs[(PT == 1 ? 0 : int64_t(U) * p.n) + int64_t(u) * p.n + st] = part[j];
      }
    }
  };
  if constexpr (PART != 2) emit(std::integral_constant<int, 1>{});
  if constexpr (PART != 1) emit(std::integral_constant<int, 2>{});
}

int blocks_for(int64_t threads) {
  return static_cast<int>((threads + kThreads - 1) / kThreads);
}

template <int ES, int D, int G>
hipError_t train_forward_impl(const TrainParams &p, hipStream_t s) {
  const int U = p.batch * p.hkv;
  const size_t states = size_t(U) * p.n * D * ES, pad = size_t(32) * D * ES;
  hipError_t e = launch_fill_u8(static_cast<char *>(p.ks) + states, pad, s);
  if (e == hipSuccess) e = launch_fill_u8(static_cast<char *>(p.vs) + states, pad, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((train_decide_kernel<ES, D>), dim3(blocks_for(int64_t(U) * p.n)), dim3(kThreads),
                     0, s, p);
  if constexpr (ES == 2) {
    const dim3 grid((p.n + 31) / 32, U);
    switch (2 + (p.window + 14) / 16) {   // 16-token k-steps for 31 + w tokens
      case 2: hipLaunchKernelGGL((train_states_mfma_kernel<D, 2>), grid, dim3(64), 0, s, p); break;
      case 3: hipLaunchKernelGGL((train_states_mfma_kernel<D, 3>), grid, dim3(64), 0, s, p); break;
      case 4: hipLaunchKernelGGL((train_states_mfma_kernel<D, 4>), grid, dim3(64), 0, s, p); break;
      case 5: hipLaunchKernelGGL((train_states_mfma_kernel<D, 5>), grid, dim3(64), 0, s, p); break;
      default: hipLaunchKernelGGL((train_states_mfma_kernel<D, 6>), grid, dim3(64), 0, s, p); break;
    }
    constexpr int TW = kWaves * (32 / G);
    const int ntiles = (p.n + TW - 1) / TW;
    hipLaunchKernelGGL((train_qmajor_kernel<D, G, 0>), dim3(8 * ((U + 7) / 8) * ntiles),
                       dim3(kThreads), 0, s, p, ntiles);
  } else {
    hipLaunchKernelGGL((train_states_kernel<ES, D>), dim3((p.n + 63) / 64, U), dim3(64), 0, s, p);
    const int ngroups = (p.n + Rows<G>::TG - 1) / Rows<G>::TG;
    hipLaunchKernelGGL((train_fwd_kernel<ES, D, G>), dim3(blocks_for(int64_t(U) * ngroups * 64)),
                       dim3(kThreads), 0, s, p, ngroups);
  }
  return hipGetLastError();
}

template <int ES, int D, int G>
hipError_t train_backward_impl(const TrainParams &p, hipStream_t s) {
  const int U = p.batch * p.hkv;
  if constexpr (ES == 2) {
    constexpr int TW = kWaves * (32 / G);
    const int ntiles = (p.n + TW - 1) / TW;
    hipLaunchKernelGGL((train_qmajor_kernel<D, G, 1>), dim3(8 * ((U + 7) / 8) * ntiles),
                       dim3(kThreads), 0, s, p, ntiles);
    const int stiles = (p.n + 127) / 128;
    hipLaunchKernelGGL((train_dkv_mfma_kernel<D, G, 1>), dim3(8 * ((U + 7) / 8) * stiles),
                       dim3(kThreads), 0, s, p, stiles);
    hipLaunchKernelGGL((train_dkv_mfma_kernel<D, G, 2>), dim3(8 * ((U + 7) / 8) * stiles),
                       dim3(kThreads), 0, s, p, stiles);
  } else {
    const int ngroups = (p.n + Rows<G>::TG - 1) / Rows<G>::TG;
    hipLaunchKernelGGL((train_dq_kernel<ES, D, G>), dim3(blocks_for(int64_t(U) * ngroups * 64)),
                       dim3(kThreads), 0, s, p, ngroups);
    const int nblocks = (p.n + 3) / 4;
    hipLaunchKernelGGL((train_dkv_kernel<ES, D, G>), dim3(blocks_for(int64_t(U) * nblocks * 64)),
                       dim3(kThreads), 0, s, p, nblocks);
  }
  if constexpr (ES == 2) {
    const dim3 grid((p.n + 31) / 32, U);
    switch (2 + (p.window + 14) / 16) {   // 16-row k-steps for the 31 + w states
      case 2: hipLaunchKernelGGL((train_tokens_mfma_kernel<D, 2>), grid, dim3(64), 0, s, p); break;
      case 3: hipLaunchKernelGGL((train_tokens_mfma_kernel<D, 3>), grid, dim3(64), 0, s, p); break;
      case 4: hipLaunchKernelGGL((train_tokens_mfma_kernel<D, 4>), grid, dim3(64), 0, s, p); break;
      case 5: hipLaunchKernelGGL((train_tokens_mfma_kernel<D, 5>), grid, dim3(64), 0, s, p); break;
      default: hipLaunchKernelGGL((train_tokens_mfma_kernel<D, 6>), grid, dim3(64), 0, s, p); break;
    }
  } else {
    hipLaunchKernelGGL((train_tokens_kernel<ES, D>), dim3((p.n + 63) / 64, U), dim3(64), 0, s, p);
  }
  hipLaunchKernelGGL((train_neurons_kernel<ES, D>), dim3(blocks_for(int64_t(U) * p.n)),
                     dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

template <int ES, int D>
hipError_t train_fwd_by_group(int group, const TrainParams &p, hipStream_t s) {
  switch (group) {
    case 1: return train_forward_impl<ES, D, 1>(p, s);
    case 2: return train_forward_impl<ES, D, 2>(p, s);
    case 4: return train_forward_impl<ES, D, 4>(p, s);
    case 8: return train_forward_impl<ES, D, 8>(p, s);
    default: return hipErrorInvalidValue;
  }
}

template <int ES, int D>
hipError_t train_bwd_by_group(int group, const TrainParams &p, hipStream_t s) {
  switch (group) {
    case 1: return train_backward_impl<ES, D, 1>(p, s);
    case 2: return train_backward_impl<ES, D, 2>(p, s);
    case 4: return train_backward_impl<ES, D, 4>(p, s);
    case 8: return train_backward_impl<ES, D, 8>(p, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_train_forward(int elem_bytes, int head_dim, int group, const TrainParams &p,
                                hipStream_t s) {
  if (elem_bytes == 2)
    return head_dim == 128 ? train_fwd_by_group<2, 128>(group, p, s) : train_fwd_by_group<2, 64>(group, p, s);
  return head_dim == 128 ? train_fwd_by_group<4, 128>(group, p, s) : train_fwd_by_group<4, 64>(group, p, s);
}

hipError_t launch_train_backward(int elem_bytes, int head_dim, int group, const TrainParams &p,
                                 hipStream_t s) {
  if (elem_bytes == 2)
    return head_dim == 128 ? train_bwd_by_group<2, 128>(group, p, s) : train_bwd_by_group<2, 64>(group, p, s);
  return head_dim == 128 ? train_bwd_by_group<4, 128>(group, p, s) : train_bwd_by_group<4, 64>(group, p, s);
}

}  // namespace dmc
