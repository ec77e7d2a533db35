// Independent Philox4x32-10 reference for the oracle's pin tests.
//
// Drives rocRAND's host-callable Philox4x32-10 engine (an implementation
// written by a third party, not by this project) and prints the raw output
// words of consecutive blocks. rocRAND keys the engine with the 64-bit seed
// and sets the 128-bit counter to (offset/4 low, offset/4 high, subsequence
// low, subsequence high), so block j of (tensor_id, step) is reached with
// subsequence = tensor_id | step << 32 and offset = 4 j.
//
// usage: rocrand_philox_ref SEED TENSOR_ID STEP FIRST_BLOCK N_BLOCKS
#include <rocrand/rocrand_kernel.h>

#include <cstdio>
#include <cstdlib>

int main(int argc, char** argv) {
  if (argc != 6) {
    std::fprintf(stderr, "usage: %s SEED TENSOR_ID STEP FIRST_BLOCK N_BLOCKS\n", argv[0]);
    return 2;
  }
  const unsigned long long seed = std::strtoull(argv[1], nullptr, 0);
  const unsigned long long tensor_id = std::strtoull(argv[2], nullptr, 0);
  const unsigned long long step = std::strtoull(argv[3], nullptr, 0);
  const unsigned long long first = std::strtoull(argv[4], nullptr, 0);
  const unsigned long long n = std::strtoull(argv[5], nullptr, 0);
  const unsigned long long subsequence = (tensor_id & 0xFFFFFFFFull) | (step << 32);
  for (unsigned long long j = first; j < first + n; ++j) {
    rocrand_state_philox4x32_10 st;
    rocrand_init(seed, subsequence, 4ull * j, &st);
    const uint4 w = rocrand4(&st);
    std::printf("%08x %08x %08x %08x\n", w.x, w.y, w.z, w.w);
  }
  return 0;
}
