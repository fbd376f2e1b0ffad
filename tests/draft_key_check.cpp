// Host check of the draft head's 64-bit (logit, id) keys, with the library's own pair_key,
// key_value and key_id compiled for the host: the unsigned order of two keys is the pair order
// (higher logit first; on equal logits, -0 and +0 included, the lower id), the key decodes to
// its logit (-0 as +0) and id, and key 0 lies below every pair. Logits are numbers (NaN never
// reaches a key). Exit status 0 and "ok <pairs>" when every case holds.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <limits>
#include <random>
#include <vector>

#include "k_draft.h"

static bool ref_better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

int main() {
  const float inf = std::numeric_limits<float>::infinity();
  const float dmin = std::numeric_limits<float>::denorm_min();
  const float fmin = std::numeric_limits<float>::min();
  const float fmax = std::numeric_limits<float>::max();
  std::vector<float> vals = {-inf, -fmax, -1e30f, -2.f, -1.f, -fmin, -dmin, -0.f, 0.f, dmin,
                             fmin, 1e-30f, 0.5f, 1.f, 1.f + 1e-7f, 2.f, 1e30f, fmax, inf};
  std::mt19937 rng(2609);
  std::uniform_int_distribution<uint32_t> bits(0, 0xffffffffu);
  while (vals.size() < 400) {
    const uint32_t u = bits(rng);
    float v;
    std::memcpy(&v, &u, 4);
    if (!std::isnan(v)) vals.push_back(v);
  }
  const std::vector<int> ids = {0, 1, 2, 31, 32000, 151935, (1 << 30) - 1};
  long pairs = 0;
  for (float va : vals)
    for (int ia : ids) {
      const uint64_t ka = asv::pair_key(va, ia);
      const float back = asv::key_value(ka);
      if (!(back == va) || std::signbit(back) != (std::signbit(va) && va != 0.f) ||
          asv::key_id(ka) != ia) {
        std::printf("decode %a id %d -> %a id %d\n", va, ia, back, asv::key_id(ka));
        return 1;
      }
      if (!(ka > 0)) {
        std::printf("key of %a id %d is not above key 0\n", va, ia);
        return 1;
      }
      for (float vb : vals)
        for (int ib : ids) {
          const uint64_t kb = asv::pair_key(vb, ib);
          if ((ka > kb) != ref_better(va, ia, vb, ib)) {
            std::printf("order (%a, %d) vs (%a, %d): keys %llx %llx\n", va, ia, vb, ib,
                        (unsigned long long)ka, (unsigned long long)kb);
            return 1;
          }
          ++pairs;
        }
    }
  std::printf("ok %ld\n", pairs);
  return 0;
}
