// Host-side cross-check of the oracle's Philox4x32-10 against rocRAND's
// open-source engine (called, not copied).  Reads "seed role idx" lines on
// stdin and prints the uniform word rocRAND yields for element idx when the
// element's block counter is (idx/4, role) -- rocrand_init(seed, role, 4*(idx/4))
// starts the engine at exactly that counter.
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>

int main() {
  unsigned long long seed, role, idx;
  while (std::scanf("%llu %llu %llu", &seed, &role, &idx) == 3) {
    rocrand_state_philox4x32_10 st;
    rocrand_init(seed, role, 4ull * (idx / 4ull), &st);
    uint4 v = rocrand4(&st);
    unsigned int w[4] = {v.x, v.y, v.z, v.w};
    std::printf("%u\n", w[idx % 4]);
  }
  return 0;
}
