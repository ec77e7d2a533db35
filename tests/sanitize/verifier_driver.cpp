// Host driver of the trusted-side verifier for sanitizer builds
// (AddressSanitizer + UndefinedBehaviorSanitizer): it runs the float32 and
// float64 recomputations over ragged float32 and bfloat16 layers, with
// several thread counts, and one run of the verifier down every path. Exits
// non-zero on a failed check; the sanitizers abort on any memory or UB error.
#include <array>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

#include "dpsgd_verifier.h"

namespace {

int failures = 0;
#define CHECK(cond)                                                       \
  do {                                                                    \
    if (!(cond)) {                                                        \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      ++failures;                                                         \
    }                                                                     \
  } while (0)

uint16_t to_bf16(float x) {
  uint32_t u;
  std::memcpy(&u, &x, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);   // round to nearest even
  return (uint16_t)(u >> 16);
}

struct Layer {
  std::vector<float> A32, G32;
  std::vector<uint16_t> A16, G16;
  dpsgd_layer d{};
};

Layer make_layer(std::mt19937& rng, int64_t B, int64_t T, int64_t d_in, int64_t d_out, int bf16,
                 uint32_t id) {
  std::normal_distribution<float> nd(0.f, 1.f);
  Layer L;
  const size_t na = (size_t)(B * T * d_in), ng = (size_t)(B * T * d_out);
  L.A32.resize(na);
  L.G32.resize(ng);
  for (auto& v : L.A32) v = nd(rng);
  for (auto& v : L.G32) v = 0.05f * nd(rng);
  if (bf16) {
    L.A16.resize(na);
    L.G16.resize(ng);
    for (size_t i = 0; i < na; ++i) L.A16[i] = to_bf16(L.A32[i]);
    for (size_t i = 0; i < ng; ++i) L.G16[i] = to_bf16(L.G32[i]);
  }
  L.d.A = bf16 ? (const void*)L.A16.data() : (const void*)L.A32.data();
  L.d.G = bf16 ? (const void*)L.G16.data() : (const void*)L.G32.data();
  L.d.B = B;
  L.d.T = T;
  L.d.d_in = d_in;
  L.d.d_out = d_out;
  L.d.dtype = bf16 ? DPSGD_BF16 : DPSGD_F32;
  L.d.tensor_id = id;
  return L;
}

void run_case(std::mt19937& rng, int64_t B, int bf16,
              const std::vector<std::array<int64_t, 3>>& dims) {
  std::vector<Layer> Ls;
  for (size_t k = 0; k < dims.size(); ++k)
    Ls.push_back(make_layer(rng, B, dims[k][0], dims[k][1], dims[k][2], bf16, (uint32_t)k));
  std::vector<dpsgd_layer> ds;
  for (auto& L : Ls) ds.push_back(L.d);
  const int n = (int)ds.size();
  std::vector<std::vector<float>> o32(n), o32b(n);
  std::vector<std::vector<double>> o64(n);
  std::vector<float*> p32(n), p32b(n);
  std::vector<double*> p64(n);
  for (int l = 0; l < n; ++l) {
    const size_t e = (size_t)(ds[l].d_out * ds[l].d_in);
    o32[l].assign(e, -1.f);
    o32b[l].assign(e, -2.f);
    o64[l].assign(e, -1.0);
    p32[l] = o32[l].data();
    p32b[l] = o32b[l].data();
    p64[l] = o64[l].data();
  }
  const float C = 0.5f;
  CHECK(dpsgd_reference_mean_f32(ds.data(), n, C, B, p32.data(), 1) == DPSGD_OK);
  CHECK(dpsgd_reference_mean_f32(ds.data(), n, C, B, p32b.data(), 3) == DPSGD_OK);
  CHECK(dpsgd_reference_mean_f64(ds.data(), n, C, B, p64.data(), 2) == DPSGD_OK);
  double nsq = 0.0, diff = 0.0, ref = 0.0;
  for (int l = 0; l < n; ++l)
    for (size_t j = 0; j < o32[l].size(); ++j) {
      CHECK(o32[l][j] == o32b[l][j]);            // independent of the thread count
      nsq += (double)o32[l][j] * o32[l][j];
      diff += (o32[l][j] - o64[l][j]) * (o32[l][j] - o64[l][j]);
      ref += o64[l][j] * o64[l][j];
    }
  CHECK(std::sqrt(nsq) <= C * (1.0 + 1e-4));      // clipped average has norm <= C
  CHECK(std::sqrt(diff) <= 1e-4 * std::sqrt(ref) + 1e-12);

  // The verifier down each path on the same layers.
  dpsgd_verifier_params pr{0.1, 1e-3, 1e-2, 0.0, 0.1, 2, (double)C, B, 1e-4};
  dpsgd_verifier_state st;
  CHECK(dpsgd_verifier_init(&pr, &st) == DPSGD_OK);
  dpsgd_verify_result r;
  std::vector<const float*> g(n);
  for (int l = 0; l < n; ++l) g[l] = o32[l].data();
  CHECK(dpsgd_verify_step(&pr, &st, ds.data(), n, g.data(), 1, 2, &r) == DPSGD_OK);
  CHECK(r.path == DPSGD_PATH_BODY && r.decision == DPSGD_VERIFY_ACCEPT);
  CHECK(dpsgd_verify_step(&pr, &st, ds.data(), n, g.data(), 0, 2, &r) == DPSGD_OK);
  CHECK(r.path == DPSGD_PATH_UNCHECKED);
  // A forged submission: the first entry moved by a few tau_abs C.
  std::vector<float> forged(o32[0]);
  forged[0] += (float)(5.0 * pr.tau_abs * C);
  g[0] = forged.data();
  CHECK(dpsgd_verify_step(&pr, &st, ds.data(), n, g.data(), 1, 2, &r) == DPSGD_OK);
  CHECK(r.path == DPSGD_PATH_AMBIGUITY || r.path == DPSGD_PATH_HARD);
  // A submission over the norm bound, and a NaN: the structural check.
  dpsgd_verifier_init(&pr, &st);
  for (auto& v : forged) v *= 1e3f;
  CHECK(dpsgd_verify_step(&pr, &st, ds.data(), n, g.data(), 0, 1, &r) == DPSGD_OK);
  CHECK(r.path == DPSGD_PATH_STRUCTURAL && st.aborted == 1);
  CHECK(dpsgd_verify_step(&pr, &st, ds.data(), n, g.data(), 0, 1, &r) == DPSGD_ERR_ABORTED);
  dpsgd_verifier_init(&pr, &st);
  forged[1] = std::nanf("");
  CHECK(dpsgd_verify_step(&pr, &st, ds.data(), n, g.data(), 1, 1, &r) == DPSGD_OK);
  CHECK(r.path == DPSGD_PATH_STRUCTURAL);
  // Invalid arguments return before touching the buffers.
  CHECK(dpsgd_reference_mean_f32(ds.data(), 0, C, B, p32.data(), 1) == DPSGD_ERR_INVALID_ARG);
  CHECK(dpsgd_reference_mean_f32(ds.data(), n, -1.f, B, p32.data(), 1) == DPSGD_ERR_INVALID_ARG);
}

}  // namespace

int main() {
  std::mt19937 rng(1234);
  run_case(rng, 3, 0, {{{5, 7, 3}}, {{5, 3, 11}}});                // float32, ragged
  run_case(rng, 4, 1, {{{17, 40, 24}}, {{17, 24, 1}}, {{17, 1, 9}}});  // bf16, one-wide
  run_case(rng, 1, 0, {{{1, 33, 65}}});                            // one example, T = 1
  run_case(rng, 2, 1, {{{130, 64, 96}}});                          // long T: Gram form
  run_case(rng, 5, 0, {{{2, 300, 200}}});                          // short T: materialised
  if (failures) {
    std::fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  std::printf("verifier driver ok\n");
  return 0;
}
