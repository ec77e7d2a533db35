// Host driver of the library's planners for sanitizer builds: the workspace
// queries, the norm-form choice and the argument checks of every entry point
// run the host-side planning code (tile counts, split plans, tail splits,
// stored-form ranges, workspace layouts) without launching a kernel. Linked
// with the library's sources built with host-only AddressSanitizer and
// UndefinedBehaviorSanitizer. Exits non-zero on a failed check.
#include <cstdio>
#include <vector>

#include "dpsgd.h"

namespace {

int failures = 0;
#define CHECK(cond)                                                       \
  do {                                                                    \
    if (!(cond)) {                                                        \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      ++failures;                                                         \
    }                                                                     \
  } while (0)

dpsgd_layer shape(int64_t B, int64_t T, int64_t d_in, int64_t d_out, int dtype, uint32_t id) {
  dpsgd_layer L{};
  L.B = B;
  L.T = T;
  L.d_in = d_in;
  L.d_out = d_out;
  L.dtype = dtype;
  L.tensor_id = id;
  return L;
}

void queries(const std::vector<dpsgd_layer>& Ls) {
  const int n = (int)Ls.size();
  for (int mode = 0; mode <= 2; ++mode) {
    const size_t nb = dpsgd_norms_workspace_bytes(Ls.data(), n, mode);
    const size_t fb = dpsgd_clipped_sum_workspace_bytes(Ls.data(), n, mode);
    CHECK(nb > 0 && nb % 256 == 0);
    CHECK(fb >= nb);
  }
  CHECK(dpsgd_clip_workspace_bytes(Ls.data(), n) >= (size_t)Ls[0].B * 4);
  for (const auto& L : Ls) {
    const int32_t m = dpsgd_select_norm_mode(&L);
    CHECK(m == DPSGD_NORM_GHOST || m == DPSGD_NORM_MATERIALIZE || m == DPSGD_NORM_CLOSED_FORM);
    CHECK((m == DPSGD_NORM_CLOSED_FORM) == (L.T == 1));
  }
  // Argument checks: NULL data pointers are refused before any planning
  // reaches a launch.
  std::vector<float> norms(1);
  CHECK(dpsgd_per_example_norms_multi(Ls.data(), n, 0, norms.data(), 0, nullptr, 0, nullptr) ==
        DPSGD_ERR_INVALID_ARG);
}

}  // namespace

int main() {
  const int BF = DPSGD_BF16, F = DPSGD_F32;
  queries({shape(32, 1, 256, 128, F, 0)});                                     // c1
  queries({shape(256, 1, 784, 512, F, 0), shape(256, 1, 512, 10, F, 1)});     // c2
  queries({shape(64, 512, 768, 3072, BF, 0)});                                 // c3
  queries({shape(16, 1024, 4096, 11008, BF, 0), shape(16, 1024, 4096, 16, BF, 1),
           shape(16, 1024, 16, 4096, BF, 2)});                                 // c4
  std::vector<dpsgd_layer> c5;
  for (int b = 0; b < 12; ++b) {
    const int64_t dims[4][2] = {{768, 2304}, {768, 768}, {768, 3072}, {3072, 768}};
    for (int k = 0; k < 4; ++k) c5.push_back(shape(128, 256, dims[k][0], dims[k][1], BF, 4 * b + k));
  }
  queries(c5);                                                                 // c5: 48 layers
  std::vector<dpsgd_layer> many;                                               // > 48 per launch
  for (int k = 0; k < 100; ++k) many.push_back(shape(3, 64 + (k % 5) * 32, 256, 384, BF, k));
  queries(many);
  std::vector<dpsgd_layer> wrn;                                                // WRN-16-4 im2col
  const int64_t conv[][3] = {{1024, 27, 16}, {1024, 144, 64}, {1024, 576, 64}, {256, 576, 128},
                             {256, 1152, 128}, {64, 1152, 256}, {64, 2304, 256}, {1, 256, 10}};
  for (int k = 0; k < 8; ++k) wrn.push_back(shape(512, conv[k][0], conv[k][1], conv[k][2], F, k));
  queries(wrn);
  queries({shape(1, 1, 1, 1, F, 0)});                                          // degenerate
  queries({shape(2, 37, 13, 21, BF, 0), shape(2, 37, 1, 33, BF, 1), shape(2, 37, 33, 1, BF, 2)});
  queries({shape(8, 128, 768, 4, F, 0), shape(8, 128, 4, 2304, F, 1)});        // adapters
  queries({shape(1 << 20, 1, 4, 4, F, 0)});                                    // many examples
  // Gram form on 256-row tiles: the park area (256 KB per workgroup) and the
  // grid cap of 512 workgroups (200 x 6 = 1200 jobs).
  const dpsgd_layer c4base = shape(16, 1024, 4096, 11008, BF, 0);
  CHECK(dpsgd_norms_workspace_bytes(&c4base, 1, DPSGD_NORM_GHOST) == 1024 + (size_t)256 * 262144);
  const dpsgd_layer capped = shape(200, 520, 64, 64, BF, 0);
  CHECK(dpsgd_norms_workspace_bytes(&capped, 1, DPSGD_NORM_GHOST) == 7424 + (size_t)512 * 262144);
  queries({capped, shape(200, 300, 128, 64, BF, 1)});
  // Ragged last row tiles of the 384x256 clip kernel, with a split tail, and
  // a 4096 x 4096 layer (one round of 256x256 tiles).
  queries({shape(1, 128, 6144, 4064, BF, 0)});
  queries({shape(2, 64, 6144, 4064, BF, 0)});
  queries({shape(16, 1024, 4096, 4096, BF, 0)});
  if (failures) {
    std::fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  std::printf("planner driver ok\n");
  return 0;
}
