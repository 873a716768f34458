// Damaged-file check of the GGUF split-pack reader (moe_pack_gguf), built with
// AddressSanitizer and UndefinedBehaviorSanitizer by tests/test_pack.py.  For each
// valid seed file: truncations at random lengths, random byte flips, and 8-byte
// fields overwritten with extreme values (0, 2^31, 2^32-1, 2^63, 2^64-1, random),
// each written to a file and packed.  Every call must return one of the
// interface's codes; a successful pack must report consistent sizes.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <string>
#include <vector>

#include "../include/moecache.h"

void moecache_set_last_error(const char *) {}  // the library's error slot, not needed here

static std::vector<uint8_t> slurp(const char *path) {
  std::vector<uint8_t> v;
  std::FILE *f = std::fopen(path, "rb");
  if (!f) return v;
  uint8_t buf[65536];
  size_t n;
  while ((n = std::fread(buf, 1, sizeof buf, f)) > 0) v.insert(v.end(), buf, buf + n);
  std::fclose(f);
  return v;
}

int main(int argc, char **argv) {
  if (argc < 3) return 2;
  const std::string dir = argv[1];
  const std::string in = dir + "/fuzz.gguf", pk = dir + "/fuzz.pack", ix = dir + "/fuzz.index",
                    rt = dir + "/fuzz.router";
  std::mt19937_64 rng(2024);
  long runs = 0, ok = 0;
  for (int s = 2; s < argc; ++s) {
    const std::vector<uint8_t> seed = slurp(argv[s]);
    if (seed.size() < 64) return 3;
    moe_pack_info info{};
    if (moe_pack_gguf(argv[s], pk.c_str(), ix.c_str(), rt.c_str(), &info) != MOE_OK) return 4;
    const uint64_t extremes[] = {0, 1ull << 31, 0xffffffffull, 1ull << 63, ~0ull, 0};
    for (int it = 0; it < 1500; ++it) {
      std::vector<uint8_t> b = seed;
      const int kind = (int)(rng() % 3);
      if (kind == 0) {
        b.resize(rng() % b.size());
      } else if (kind == 1) {
        const int flips = 1 + (int)(rng() % 8);
        for (int i = 0; i < flips; ++i) b[rng() % b.size()] ^= (uint8_t)(1u << (rng() % 8));
      } else {
        // overwrite an 8-byte field, most often inside the header / metadata / tensor infos
        const size_t span = std::min<size_t>(b.size() - 8, 4096);
        const size_t at = rng() % span;
        uint64_t v = extremes[rng() % 6];
        if (v == 0 && rng() % 2) v = rng();
        std::memcpy(&b[at], &v, 8);
      }
      std::FILE *f = std::fopen(in.c_str(), "wb");
      if (!f) return 5;
      if (!b.empty() && std::fwrite(b.data(), 1, b.size(), f) != b.size()) return 6;
      std::fclose(f);
      moe_pack_info o{};
      const int rc = moe_pack_gguf(in.c_str(), pk.c_str(), ix.c_str(), rt.c_str(), &o);
      ++runs;
      if (rc == MOE_OK) {
        ++ok;
        if (o.pack_bytes != (uint64_t)o.n_layers * o.n_experts * o.payload_bytes) {
          std::printf("inconsistent sizes at iteration %d\n", it);
          return 7;
        }
      } else if (rc != MOE_EINVAL && rc != MOE_EIO && rc != MOE_ENOMEM) {
        std::printf("unexpected code %d at iteration %d\n", rc, it);
        return 8;
      }
    }
  }
  std::printf("ok %ld runs, %ld packed\n", runs, ok);
  return 0;
}
