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
// These are vector-ALU kernels (lanes own head-dim elements, one wave per
// group of rows); they work for every dtype.
#include "dmc_device.h"

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
  L.ks = take(U * N * D * elem_bytes);
  L.vs = take(U * N * D * elem_bytes);
  L.x = take(U * N * 4);
  L.alpha = take(U * N * 4);
  L.omega = take(U * N * 4);
  L.z = take(U * N * 4);
  L.mask = take(U * N * 4);
  L.lse = take(U * G * N * 4);
  L.dsum = take(U * G * N * 4);
  L.dks = take(U * N * D * 4);
  L.dvs = take(U * N * D * 4);
  L.dmask = take(U * N * 4);
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

// Per token: Gumbel-sigmoid logit, alpha, omega; the mask entry of the
// previous state (log(1 - alpha_t) belongs to state t - 1).
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
  p.x[i] = x;
  p.alpha[i] = al;
  p.omega[i] = om;
  if (p.alpha_out) p.alpha_out[(int64_t(b) * p.n + t) * p.hkv + g] = al;
  if (t > 0) p.mask[i - 1] = log_one_minus_sigmoid(x);
  if (t == p.n - 1) p.mask[i] = 0.0f;   // the last state has no successor
}

// Unrolled states, one wave per (unit, 64 positions): state j is the
// closed-form partial accumulation over its window, walked from j down to
// the window start with the running product of alphas.
template <int ES, int D>
__global__ __launch_bounds__(64) void train_states_kernel(TrainParams p) {
  constexpr int E = D / 64, kB = 4;
  const int u = blockIdx.y, lane = threadIdx.x;
  const int b = u / p.hkv, g = u - b * p.hkv;
  const int j0 = blockIdx.x * 64, j1 = min(j0 + 64, p.n);
  const float *al = p.alpha + int64_t(u) * p.n;
  const float *om = p.omega + int64_t(u) * p.n;
  const char *kb = static_cast<const char *>(p.k) + (row_k(p, b, 0, g, D) + lane * E) * ES;
  const char *vb = static_cast<const char *>(p.v) + (row_k(p, b, 0, g, D) + lane * E) * ES;
  const int64_t rs = int64_t(p.hkv) * D * ES;   // bytes between tokens
  for (int j = j0; j < j1; ++j) {
    const int a = max(0, j - p.window + 1);
    float sk[E], sv[E], zs = 0.0f, P = 1.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) sk[e] = sv[e] = 0.0f;
    for (int t0 = j; t0 >= a; t0 -= kB) {
      float kk[kB][E], vv[kB][E], wa[kB], wo[kB];
#pragma unroll
      for (int q = 0; q < kB; ++q) {
        const int t = max(t0 - q, a);
        load_e<ES, E>(kb + t * rs, kk[q]);
        load_e<ES, E>(vb + t * rs, vv[q]);
        wa[q] = al[t];
        wo[q] = om[t];
      }
#pragma unroll
      for (int q = 0; q < kB; ++q) {
        if (t0 - q < a) break;
        if (lane == 0) kk[q][0] = 0.0f;   // k_t[0] <- 0
        const float c = wo[q] * P;        // omega_t * prod_{r = t+1 .. j} alpha_r
#pragma unroll
        for (int e = 0; e < E; ++e) {
          sk[e] = fmaf(c, kk[q][e], sk[e]);
          sv[e] = fmaf(c, vv[q][e], sv[e]);
        }
        zs += c;
        P *= wa[q];
      }
    }
    const float inv = 1.0f / zs;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      sk[e] *= inv;
      sv[e] *= inv;
    }
    const int64_t o = (int64_t(u) * p.n + j) * D + lane * E;
    store_e<ES, E>(static_cast<char *>(p.ks) + o * ES, sk);
    store_e<ES, E>(static_cast<char *>(p.vs) + o * ES, sv);
    if (lane == 0) p.z[int64_t(u) * p.n + j] = zs;
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
    if (lane == 0) p.lse[(int64_t(u) * G + h) * p.n + a + j] = m[r] + __log2f(l[r]);
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
      Lr[r] = p.lse[(int64_t(u) * G + h) * p.n + a + j];
      if (lane == 0) p.dsum[(int64_t(u) * G + h) * p.n + a + j] = Dr[r];
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
      const float L = p.lse[(int64_t(u) * G + h) * p.n + t];
      const float Dt = p.dsum[(int64_t(u) * G + h) * p.n + t];
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

// States -> tokens, part 1, one wave per (unit, 64 tokens): token t feeds
// states j = t .. t + w - 1 with weight c_tj / z_j; its key and value
// gradients gather those states' gradients, and e_tj = d loss / d c_tj =
// ((k^_t - K~_j) . dK~_j + (v_t - V~_j) . dV~_j) / z_j is kept for part 2.
template <int ES, int D>
__global__ __launch_bounds__(64) void train_tokens_kernel(TrainParams p) {
  constexpr int E = D / 64;
  const int u = blockIdx.y, lane = threadIdx.x;
  const int b = u / p.hkv, g = u - b * p.hkv;
  const int t0 = blockIdx.x * 64, t1 = min(t0 + 64, p.n);
  const float *al = p.alpha + int64_t(u) * p.n;
  const float *om = p.omega + int64_t(u) * p.n;
  const float *zz = p.z + int64_t(u) * p.n;
  for (int t = t0; t < t1; ++t) {
    const int64_t ro = row_k(p, b, t, g, D) + lane * E;
    float kt[E], vt[E];
    load_e<ES, E>(static_cast<const char *>(p.k) + ro * ES, kt);
    load_e<ES, E>(static_cast<const char *>(p.v) + ro * ES, vt);
    if (lane == 0) kt[0] = 0.0f;
    float dk[E], dv[E], P = 1.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) dk[e] = dv[e] = 0.0f;
    const int jl = min(t + p.window - 1, p.n - 1);
    for (int j = t; j <= jl; ++j) {
      if (j > t) P *= al[j];
      const float zj = zz[j];
      const float cz = om[t] * P / zj;
      const int64_t so = (int64_t(u) * p.n + j) * D + lane * E;
      float ks[E], vs[E], dks[E], dvs[E];
      load_e<ES, E>(static_cast<const char *>(p.ks) + so * ES, ks);
      load_e<ES, E>(static_cast<const char *>(p.vs) + so * ES, vs);
      float ev = 0.0f;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        dks[e] = p.dks[so + e];
        dvs[e] = p.dvs[so + e];
        dk[e] = fmaf(cz, dks[e], dk[e]);
        dv[e] = fmaf(cz, dvs[e], dv[e]);
        ev = fmaf(kt[e] - ks[e], dks[e], ev);
        ev = fmaf(vt[e] - vs[e], dvs[e], ev);
      }
      ev = wsum(ev) / zj;
      if (lane == 0) p.e[(int64_t(u) * p.n + t) * p.window + (j - t)] = ev;
    }
    if (lane == 0) dk[0] = 0.0f;   // element 0 gets the decision gradient in part 2
    store_e<ES, E>(static_cast<char *>(p.dk) + ro * ES, dk);
    store_e<ES, E>(static_cast<char *>(p.dv) + ro * ES, dv);
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

int blocks_for(int64_t threads) {
  return static_cast<int>((threads + kThreads - 1) / kThreads);
}

template <int ES, int D, int G>
hipError_t train_forward_impl(const TrainParams &p, hipStream_t s) {
  const int U = p.batch * p.hkv;
  hipLaunchKernelGGL((train_decide_kernel<ES, D>), dim3(blocks_for(int64_t(U) * p.n)), dim3(kThreads),
                     0, s, p);
  hipLaunchKernelGGL((train_states_kernel<ES, D>), dim3((p.n + 63) / 64, U), dim3(64), 0, s, p);
  const int ngroups = (p.n + Rows<G>::TG - 1) / Rows<G>::TG;
  hipLaunchKernelGGL((train_fwd_kernel<ES, D, G>), dim3(blocks_for(int64_t(U) * ngroups * 64)),
                     dim3(kThreads), 0, s, p, ngroups);
  return hipGetLastError();
}

template <int ES, int D, int G>
hipError_t train_backward_impl(const TrainParams &p, hipStream_t s) {
  const int U = p.batch * p.hkv;
  const int ngroups = (p.n + Rows<G>::TG - 1) / Rows<G>::TG;
  hipLaunchKernelGGL((train_dq_kernel<ES, D, G>), dim3(blocks_for(int64_t(U) * ngroups * 64)),
                     dim3(kThreads), 0, s, p, ngroups);
  const int nblocks = (p.n + 3) / 4;
  hipLaunchKernelGGL((train_dkv_kernel<ES, D, G>), dim3(blocks_for(int64_t(U) * nblocks * 64)),
                     dim3(kThreads), 0, s, p, nblocks);
  hipLaunchKernelGGL((train_tokens_kernel<ES, D>), dim3((p.n + 63) / 64, U), dim3(64), 0, s, p);
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
