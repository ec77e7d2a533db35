// Trusted-side verifier of DP-SGD submissions (host C++, no GPU runtime).
//
// Paper: Section "Two-Stage Verification", algorithm "TEE Verification", and
// the clipped average of Section 2.2. The recomputation is the verifier's own
// float32 / float64 implementation of the clipped average. A step is first
// classified from the thresholds (structural, unchecked, body, hard or
// ambiguity), then charged to the one ledger of its class.
//
// Determinism: every reduction has a fixed order that does not depend on the
// thread count. Squared norms are per example (one task per example, layers
// in order); dot products use eight interleaved partial sums combined in a
// fixed order (so they vectorise); the weighted sum of an output element runs
// over the B*T rows in increasing order, in fixed groups (see weighted_sum).
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <limits>
#include <thread>
#include <vector>

#include "dpsgd_verifier.h"

namespace {

inline float bf16_to_f32(uint16_t h) {
  const uint32_t u = (uint32_t)h << 16;
  float f;
  std::memcpy(&f, &u, sizeof f);
  return f;
}

template <typename T>
void load_row(int dtype, const void* base, int64_t row, int64_t width, T* dst) {
  if (dtype == DPSGD_BF16) {
    const uint16_t* p = static_cast<const uint16_t*>(base) + row * width;
    for (int64_t j = 0; j < width; ++j) dst[j] = (T)bf16_to_f32(p[j]);
  } else {
    const float* p = static_cast<const float*>(base) + row * width;
    for (int64_t j = 0; j < width; ++j) dst[j] = (T)p[j];
  }
}

// x . y with eight interleaved partial sums, combined pairwise in a fixed order.
template <typename T>
T dot(const T* x, const T* y, int64_t n) {
  T s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  int64_t j = 0;
  for (; j + 8 <= n; j += 8)
    for (int u = 0; u < 8; ++u) s[u] += x[j + u] * y[j + u];
  for (int u = 0; j < n; ++j, ++u) s[u] += x[j] * y[j];
  return ((s[0] + s[4]) + (s[2] + s[6])) + ((s[1] + s[5]) + (s[3] + s[7]));
}

int resolve_threads(int threads) {
  if (threads > 0) return threads;
  const unsigned h = std::thread::hardware_concurrency();
  return h ? (int)h : 1;
}

// Runs f(task) for task in [0, n) on `threads` workers (dynamic assignment;
// each task's result must not depend on which worker runs it).
template <typename F>
void parallel_tasks(int64_t n, int threads, F f) {
  const int w = (int)std::min<int64_t>(std::max(1, threads), std::max<int64_t>(n, 1));
  std::atomic<int64_t> next{0};
  auto run = [&]() {
    for (int64_t t; (t = next.fetch_add(1)) < n;) f(t);
  };
  if (w <= 1) {
    run();
    return;
  }
  std::vector<std::thread> pool;
  pool.reserve(w - 1);
  for (int k = 0; k < w - 1; ++k) pool.emplace_back(run);
  run();
  for (auto& th : pool) th.join();
}

bool layers_ok(const dpsgd_layer* layers, int n) {
  if (!layers || n < 1) return false;
  for (int l = 0; l < n; ++l) {
    const dpsgd_layer& L = layers[l];
    if (!L.A || !L.G || L.B < 1 || L.T < 1 || L.d_in < 1 || L.d_out < 1) return false;
    if (L.B != layers[0].B) return false;
    if (L.B > (INT64_C(1) << 40) / L.T) return false;
  }
  return true;
}

// Squared Frobenius norm of G_i^T A_i for example i of layer L: the Gram form
// sum_{t,s} (a_t . a_s)(g_t . g_s) when it needs fewer multiply-adds than
// materialising the d_out x d_in gradient, else the materialised gradient.
template <typename T>
T layer_norm_sq(const dpsgd_layer& L, int64_t i, std::vector<T>& a, std::vector<T>& g,
                std::vector<T>& work) {
  const int64_t Tn = L.T, di = L.d_in, dn = L.d_out;
  a.resize((size_t)(Tn * di));
  g.resize((size_t)(Tn * dn));
  for (int64_t t = 0; t < Tn; ++t) {
    load_row(L.dtype, L.A, i * Tn + t, di, &a[(size_t)(t * di)]);
    load_row(L.dtype, L.G, i * Tn + t, dn, &g[(size_t)(t * dn)]);
  }
  const double gram_cost = 0.5 * (double)Tn * (double)(Tn + 1) * (double)(di + dn);
  const double mat_cost = (double)Tn * (double)di * (double)dn + (double)di * (double)dn;
  if (gram_cost <= mat_cost) {
    T diag = 0, off = 0;
    for (int64_t t = 0; t < Tn; ++t) {
      const T* at = &a[(size_t)(t * di)];
      const T* gt = &g[(size_t)(t * dn)];
      for (int64_t s = 0; s < t; ++s)
        off += dot(at, &a[(size_t)(s * di)], di) * dot(gt, &g[(size_t)(s * dn)], dn);
      diag += dot(at, at, di) * dot(gt, gt, dn);
    }
    return diag + (T)2 * off;
  }
  work.assign((size_t)(dn * di), (T)0);
  for (int64_t t = 0; t < Tn; ++t) {
    const T* at = &a[(size_t)(t * di)];
    for (int64_t m = 0; m < dn; ++m) {
      const T gm = g[(size_t)(t * dn + m)];
      T* row = &work[(size_t)(m * di)];
      for (int64_t n = 0; n < di; ++n) row[n] += gm * at[n];
    }
  }
  return dot(work.data(), work.data(), dn * di);
}

// Weighted sum out = (1/B) W^T A over k = 0..K-1 with W[k][m] = c_{k/T} G[k][m]:
// the rows are converted (and weighted) chunk by chunk into zero-padded
// buffers; one task owns a kMB x kNB block of the output and keeps it in a
// local array across chunks. Inside a chunk a 4 x NR register block sums
// kKC consecutive rows before it is added to the block, so an output
// element's sum has one fixed order: rows in increasing order, grouped by
// kKC and by chunk.
constexpr int64_t kMB = 32;       // output rows per task
constexpr int64_t kNB = 64;       // output columns per task
constexpr int64_t kKC = 128;      // rows summed in registers
constexpr int64_t kChunk = 4096;  // rows converted per pass (multiple of kKC)

// Register block: 4 rows x 2 vectors of 32 bytes (16 floats or 8 doubles).
template <typename T>
struct RegBlock {
  typedef T vec __attribute__((vector_size(32)));
  static constexpr int VL = 32 / sizeof(T);   // lanes per vector
  static constexpr int NR = 2 * VL;           // columns of the register block
};

template <typename T>
void micro_block(const T* W, int64_t ldw, const T* A, int64_t lda, int64_t kc, T* out,
                 int64_t ldo) {
  typedef typename RegBlock<T>::vec vec;
  constexpr int VL = RegBlock<T>::VL;
  vec r[4][2];
  for (int i = 0; i < 4; ++i) r[i][0] = r[i][1] = vec{};
  for (int64_t k = 0; k < kc; ++k) {
    vec a0, a1;
    std::memcpy(&a0, A + k * lda, sizeof a0);
    std::memcpy(&a1, A + k * lda + VL, sizeof a1);
    const T* w = W + k * ldw;
    for (int i = 0; i < 4; ++i) {
      const vec wi = vec{} + w[i];
      r[i][0] += wi * a0;
      r[i][1] += wi * a1;
    }
  }
  for (int i = 0; i < 4; ++i)
    for (int h = 0; h < 2; ++h) {
      vec o;
      std::memcpy(&o, out + i * ldo + h * VL, sizeof o);
      o += r[i][h];
      std::memcpy(out + i * ldo + h * VL, &o, sizeof o);
    }
}

template <typename T>
void weighted_sum(const dpsgd_layer& L, const T* c, T inv_b, T* out, int threads) {
  const int64_t di = L.d_in, dn = L.d_out, K = L.B * L.T;
  const int64_t tiles_m = (dn + kMB - 1) / kMB, tiles_n = (di + kNB - 1) / kNB;
  const int64_t dip = tiles_n * kNB, dnp = tiles_m * kMB;
  std::vector<T> acc((size_t)(dnp * dip), (T)0);
  // Converted rows in panel-major order: panel p of A holds columns
  // [p kNB, (p + 1) kNB) of every row of the chunk contiguously (row stride
  // kNB), and likewise for the weighted G with kMB columns, so the register
  // block walks its rows at a short fixed stride.
  const int64_t rows = std::min(kChunk, (K + kKC - 1) / kKC * kKC);
  std::vector<T> Ab((size_t)(rows * dip)), Wb((size_t)(rows * dnp));
  for (int64_t k0 = 0; k0 < K; k0 += kChunk) {
    const int64_t kn = std::min(kChunk, K - k0);
    const int64_t knp = (kn + kKC - 1) / kKC * kKC;
    parallel_tasks(knp, threads, [&](int64_t r) {
      std::vector<T> arow((size_t)dip, (T)0), wrow((size_t)dnp, (T)0);
      if (r < kn) {
        load_row(L.dtype, L.A, k0 + r, di, arow.data());
        load_row(L.dtype, L.G, k0 + r, dn, wrow.data());
        const T ck = c[(size_t)((k0 + r) / L.T)];
        for (int64_t m = 0; m < dn; ++m) wrow[(size_t)m] = ck * wrow[(size_t)m];
      }
      for (int64_t p = 0; p < tiles_n; ++p)
        std::memcpy(&Ab[(size_t)((p * knp + r) * kNB)], &arow[(size_t)(p * kNB)], kNB * sizeof(T));
      for (int64_t p = 0; p < tiles_m; ++p)
        std::memcpy(&Wb[(size_t)((p * knp + r) * kMB)], &wrow[(size_t)(p * kMB)], kMB * sizeof(T));
    });
    parallel_tasks(tiles_m * tiles_n, threads, [&](int64_t t) {
      const int64_t pm = t / tiles_n, pn = t % tiles_n;
      const T* Wp = &Wb[(size_t)(pm * knp * kMB)];
      const T* Ap = &Ab[(size_t)(pn * knp * kNB)];
      T* o = &acc[(size_t)(pm * kMB * dip + pn * kNB)];
      constexpr int NR = RegBlock<T>::NR;
      for (int64_t kc = 0; kc < knp; kc += kKC)
        for (int64_t mr = 0; mr < kMB; mr += 4)
          for (int64_t nr = 0; nr < kNB; nr += NR)
            micro_block<T>(Wp + kc * kMB + mr, kMB, Ap + kc * kNB + nr, kNB, kKC,
                           o + mr * dip + nr, dip);
    });
  }
  for (int64_t m = 0; m < dn; ++m)
    for (int64_t n = 0; n < di; ++n) out[m * di + n] = acc[(size_t)(m * dip + n)] * inv_b;
}

template <typename T>
int reference_mean(const dpsgd_layer* layers, int n_layers, T C, int64_t Bden, T* const* out,
                   int threads) {
  if (!layers_ok(layers, n_layers) || !out || Bden < 1 || !(C > (T)0)) return DPSGD_ERR_INVALID_ARG;
  for (int l = 0; l < n_layers; ++l) {
    if (!out[l]) return DPSGD_ERR_INVALID_ARG;
    if (layers[l].dtype != DPSGD_F32 && layers[l].dtype != DPSGD_BF16) return DPSGD_ERR_UNSUPPORTED;
    if (layers[l].dtype != layers[0].dtype) return DPSGD_ERR_UNSUPPORTED;
  }
  threads = resolve_threads(threads);
  const int64_t B = layers[0].B;

  // Per-example squared norms over all layers (one task per example and
  // layer, summed over layers in order), then c_i = min(1, C / n_i).
  std::vector<T> part((size_t)(B * n_layers));
  parallel_tasks(B * n_layers, threads, [&](int64_t task) {
    std::vector<T> a, g, work;
    const int64_t i = task / n_layers;
    const int l = (int)(task % n_layers);
    part[(size_t)task] = layer_norm_sq<T>(layers[l], i, a, g, work);
  });
  std::vector<T> c((size_t)B);
  for (int64_t i = 0; i < B; ++i) {
    T nsq = 0;
    for (int l = 0; l < n_layers; ++l) nsq += part[(size_t)(i * n_layers + l)];
    const T n = std::sqrt(nsq);
    c[(size_t)i] = n > (T)0 ? std::min((T)1, C / n) : (T)1;
  }

  const T inv_b = (T)1 / (T)Bden;
  for (int l = 0; l < n_layers; ++l) weighted_sum<T>(layers[l], c.data(), inv_b, out[l], threads);
  return DPSGD_OK;
}

bool params_ok(const dpsgd_verifier_params* p) {
  if (!p) return false;
  auto nonneg = [](double x) { return x >= 0.0 && std::isfinite(x); };
  return p->C > 0.0 && std::isfinite(p->C) && p->B >= 1 && nonneg(p->tau_abs) &&
         nonneg(p->rho_amb) && nonneg(p->rho_ill) && nonneg(p->K_sub) && p->K_amb >= 0 &&
         nonneg(p->norm_slack) && p->p >= 0.0 && p->p <= 1.0 &&
         (p->rho_amb > 0.0 || p->rho_ill > 0.0);
}

// ||g - ref||_2 over all layers, where ref is the verifier's own clipped
// average recomputed in T (float or double). *status receives the
// recomputation's status.
template <typename T>
double distance_to_reference(const dpsgd_layer* layers, int n, const float* const* g, double C,
                             int64_t B, int threads, int* status) {
  std::vector<std::vector<T>> ref((size_t)n);
  std::vector<T*> ptr((size_t)n);
  for (int l = 0; l < n; ++l) {
    ref[(size_t)l].resize((size_t)(layers[l].d_out * layers[l].d_in));
    ptr[(size_t)l] = ref[(size_t)l].data();
  }
  *status = reference_mean<T>(layers, n, (T)C, B, ptr.data(), threads);
  if (*status != DPSGD_OK) return 0.0;
  double s = 0.0;
  for (int l = 0; l < n; ++l) {
    const int64_t e = layers[l].d_out * layers[l].d_in;
    for (int64_t j = 0; j < e; ++j) {
      const double d = (double)g[l][j] - (double)ref[(size_t)l][(size_t)j];
      s += d * d;
    }
  }
  return std::sqrt(s);
}

}  // namespace

extern "C" {

int dpsgd_verifier_init(const dpsgd_verifier_params* params, dpsgd_verifier_state* state) {
  if (!params_ok(params) || !state) return DPSGD_ERR_INVALID_ARG;
  std::memset(state, 0, sizeof *state);
  return DPSGD_OK;
}

int dpsgd_reference_mean_f32(const dpsgd_layer* layers, int n_layers, float C, int64_t B,
                             float* const* out, int threads) {
  return reference_mean<float>(layers, n_layers, C, B, out, threads);
}

int dpsgd_reference_mean_f64(const dpsgd_layer* layers, int n_layers, double C, int64_t B,
                             double* const* out, int threads) {
  return reference_mean<double>(layers, n_layers, C, B, out, threads);
}

int dpsgd_verify_step(const dpsgd_verifier_params* params, dpsgd_verifier_state* state,
                      const dpsgd_layer* layers, int n_layers, const float* const* g_gpu, int coin,
                      int threads, dpsgd_verify_result* result) {
  if (!params_ok(params) || !state || !result || !g_gpu || !layers_ok(layers, n_layers))
    return DPSGD_ERR_INVALID_ARG;
  for (int l = 0; l < n_layers; ++l)
    if (!g_gpu[l]) return DPSGD_ERR_INVALID_ARG;
  if (state->aborted) return DPSGD_ERR_ABORTED;
  const double nan = std::numeric_limits<double>::quiet_NaN();
  dpsgd_verify_result r{DPSGD_VERIFY_ACCEPT, DPSGD_PATH_UNCHECKED, 0.0, nan, nan};
  const double C = params->C;
  // Each bound below accepts only a value within it, so NaN never passes.
  auto within = [](double v, double bound) { return v <= bound; };

  // 1. Classify the step. The norm bound holds for every honest clipped
  //    average, so it is tested on every submission, before the coin.
  double nsq = 0.0;
  for (int l = 0; l < n_layers; ++l) {
    const int64_t e = layers[l].d_out * layers[l].d_in;
    for (int64_t j = 0; j < e; ++j) nsq += (double)g_gpu[l][j] * (double)g_gpu[l][j];
  }
  r.norm = std::sqrt(nsq);
  int path;
  if (!within(r.norm, C * (1.0 + params->norm_slack))) {
    path = DPSGD_PATH_STRUCTURAL;
  } else if (!coin) {
    path = DPSGD_PATH_UNCHECKED;
  } else {
    int st = DPSGD_OK;
    r.z32 = distance_to_reference<float>(layers, n_layers, g_gpu, C, params->B, threads, &st) / C;
    if (st != DPSGD_OK) return st;
    if (within(r.z32, params->tau_abs)) {
      path = DPSGD_PATH_BODY;
    } else if (params->rho_amb > 0.0) {
      // Escalation to the float64 recomputation, in the accountant's units.
      r.n_t = (double)params->B / (2.0 * C) *
              distance_to_reference<double>(layers, n_layers, g_gpu, C, params->B, threads, &st);
      if (st != DPSGD_OK) return st;
      path = within(r.n_t, params->rho_amb * (double)params->B / 2.0) ? DPSGD_PATH_AMBIGUITY
                                                                      : DPSGD_PATH_HARD;
    } else {
      // A family without the float64 layer: a hard cap on z32 instead.
      path = within(r.z32, params->rho_ill) ? DPSGD_PATH_AMBIGUITY : DPSGD_PATH_HARD;
    }
  }

  // 2. One ledger update for the class, and the decision.
  ++state->steps;
  bool abort = path == DPSGD_PATH_STRUCTURAL || path == DPSGD_PATH_HARD;
  if (path != DPSGD_PATH_STRUCTURAL && path != DPSGD_PATH_UNCHECKED) ++state->checked;
  if (path == DPSGD_PATH_BODY) {
    state->Z_sub += r.z32;
    abort = state->Z_sub > params->K_sub;
  } else if (path == DPSGD_PATH_AMBIGUITY) {
    ++state->S_amb;
    abort = state->S_amb > params->K_amb;
  }
  r.path = path;
  r.decision = abort ? DPSGD_VERIFY_ABORT : DPSGD_VERIFY_ACCEPT;
  if (abort) state->aborted = 1;
  *result = r;
  return DPSGD_OK;
}

}  // extern "C"
