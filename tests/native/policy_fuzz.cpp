// Seeded mutation fuzzer of the host side of the PASK C ABI, built on the CPU
// with AddressSanitizer and UndefinedBehaviorSanitizer (tests/test_native_fuzz.py).
//
// pask_policy_load parses untrusted bytes.  Starting from valid blobs given
// on the command line, each round mutates a copy (bit flips, byte writes,
// header fields, truncation, extension), half of the time restores the
// trailing FNV-1a hash so that the mutation reaches the checks behind it, and
// loads it from a heap buffer of exactly its size (a read past the end is an
// ASan error).  A blob that loads must satisfy the parsed table's invariants.
// The geometry checks (pask_cache_layout_query, pask_cache_bytes,
// pask_workspace_bytes) get random geometries too.
//
// The kernels are not linked: this file defines the launchers the C ABI calls
// and the two HIP runtime calls it makes, as stubs that must never run (the
// fuzzed calls fail or return before any of them).
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "pask_internal.h"

namespace pask {
static void never(const char* what) {
  fprintf(stderr, "fuzz: %s reached (no HIP call may run here)\n", what);
  abort();
}
hipError_t launch_reset(const CacheView&, int32_t, hipStream_t) { never("launch_reset"); return hipSuccess; }
hipError_t launch_append(const AppendArgs&, hipStream_t) { never("launch_append"); return hipSuccess; }
hipError_t launch_append_step(const AppendArgs&, hipStream_t) { never("launch_append_step"); return hipSuccess; }
hipError_t launch_budget_init(const CacheView&, int32_t, int64_t, hipStream_t) { never("budget"); return hipSuccess; }
hipError_t launch_attention(const AttnArgs&, int, hipStream_t) { never("launch_attention"); return hipSuccess; }
hipError_t launch_distortion(const AttnArgs&, const AttnArgs&, int, const uint8_t*, float*, hipStream_t) {
  never("launch_distortion");
  return hipSuccess;
}
hipError_t scratch_workspace(void**) { never("scratch_workspace"); return hipSuccess; }
}  // namespace pask

extern "C" hipError_t hipMemcpyAsync(void*, const void*, size_t, hipMemcpyKind, hipStream_t) {
  pask::never("hipMemcpyAsync");
  return hipSuccess;
}
extern "C" hipError_t hipStreamSynchronize(hipStream_t) {
  pask::never("hipStreamSynchronize");
  return hipSuccess;
}
extern "C" hipError_t hipStreamIsCapturing(hipStream_t, hipStreamCaptureStatus*) {
  pask::never("hipStreamIsCapturing");
  return hipSuccess;
}
extern "C" hipError_t hipGetLastError(void) {
  pask::never("hipGetLastError");
  return hipSuccess;
}
extern "C" const char* hipGetErrorString(hipError_t) {
  pask::never("hipGetErrorString");
  return "";
}

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint64_t next_u64() {   // xorshift64*
  g_state ^= g_state >> 12;
  g_state ^= g_state << 25;
  g_state ^= g_state >> 27;
  return g_state * 0x2545F4914F6CDD1Dull;
}
uint32_t below(uint32_t n) { return n ? (uint32_t)(next_u64() % n) : 0u; }

uint32_t fnv1a(const uint8_t* d, size_t n) {
  uint32_t h = 0x811C9DC5u;
  for (size_t i = 0; i < n; ++i) {
    h ^= d[i];
    h *= 0x01000193u;
  }
  return h;
}

std::vector<uint8_t> read_file(const char* path) {
  std::vector<uint8_t> out;
  FILE* f = fopen(path, "rb");
  if (!f) return out;
  uint8_t buf[4096];
  size_t n;
  while ((n = fread(buf, 1, sizeof(buf), f)) > 0) out.insert(out.end(), buf, buf + n);
  fclose(f);
  return out;
}

void mutate(std::vector<uint8_t>& b) {
  const int n_mut = 1 + (int)below(4);
  for (int m = 0; m < n_mut; ++m) {
    switch (below(7)) {
      case 0: if (!b.empty()) b[below((uint32_t)b.size())] ^= (uint8_t)(1u << below(8)); break;
      case 1: if (!b.empty()) b[below((uint32_t)b.size())] = (uint8_t)next_u64(); break;
      case 2: {   // a header word (counts, sizes, version) to an edge value
        static const uint32_t edge[] = {0u, 1u, 2u, 3u, 6u, 12u, 16u, 17u, 63u, 64u, 65u, 128u, 129u,
                                        0x7FFFFFFFu, 0xFFFFFFFFu, 0x80000000u, 36u};
        const uint32_t v = edge[below(sizeof(edge) / sizeof(edge[0]))];
        const uint32_t off = 4 * below(8);
        if (b.size() >= off + 4) memcpy(&b[off], &v, 4);
        break;
      }
      case 3: if (!b.empty()) b.resize(below((uint32_t)b.size())); break;
      case 4: { const uint32_t k = 1 + below(64); for (uint32_t i = 0; i < k; ++i) b.push_back((uint8_t)next_u64()); break; }
      case 5: {   // the controller section's n_states / a float of rho to an edge value
        if (b.size() < 48) break;
        const uint32_t off = 32 + 4 * below((uint32_t)(b.size() - 36) / 4);
        static const uint32_t fv[] = {0x7F800000u, 0xFF800000u, 0x7FC00000u, 0x80000000u, 0xBF800000u, 65u, 64u, 0u};
        const uint32_t v = fv[below(sizeof(fv) / sizeof(fv[0]))];
        memcpy(&b[off], &v, 4);
        break;
      }
      default: if (b.size() > 1) { const uint32_t i = below((uint32_t)b.size()), j = below((uint32_t)b.size()); std::swap(b[i], b[j]); }
    }
  }
  if (below(2) && b.size() >= 4) {   // restore the hash so the later checks run
    const uint32_t h = fnv1a(b.data(), b.size() - 4);
    memcpy(&b[b.size() - 4], &h, 4);
  }
}

bool table_ok(const pask_policy& p) {
  if (p.n_tags < 1 || p.n_tags > PASK_MAX_TAGS || p.n_groups < 1 || p.n_groups > PASK_MAX_GROUPS) return false;
  if (p.n_layers < 1 || p.n_layers > PASK_MAX_LAYERS || p.n_states > PASK_MAX_STATES) return false;
  for (uint32_t l = 0; l < p.n_layers; ++l)
    if (p.group_of_layer[l] >= p.n_groups) return false;
  for (uint32_t z = 0; z < p.n_tags; ++z)
    for (uint32_t c = 0; c < p.n_groups; ++c) {
      if (p.action[z][c] > 2 || p.floor_[z][c] > 2) return false;
      for (int k = 0; k < 2; ++k) {
        const float r = p.rho_up[z][c][k];
        if (!(r >= 0.0f) || r > 3.4e38f) return false;
      }
    }
  for (uint32_t s = 0; s < p.n_states; ++s)
    if (p.crit[s] > 1) return false;
  return true;
}

pask_geom random_geom() {
  pask_geom g;
  int32_t* w = reinterpret_cast<int32_t*>(&g);
  static const int32_t edge[] = {0, 1, 2, 4, 8, 16, 32, 64, 128, 129, 65535, 65536, -1, 1 << 28, (1 << 28) + 1,
                                 0x7FFFFFFF, (int32_t)0x80000000};
  for (size_t i = 0; i < sizeof(g) / 4; ++i) w[i] = below(3) ? edge[below(sizeof(edge) / sizeof(edge[0]))] : (int32_t)next_u64();
  return g;
}

}  // namespace

int main(int argc, char** argv) {
  if (argc < 4) {
    fprintf(stderr, "usage: policy_fuzz SEED ROUNDS blob...\n");
    return 2;
  }
  g_state ^= strtoull(argv[1], nullptr, 10) * 0x9E3779B97F4A7C15ull;
  const long rounds = strtol(argv[2], nullptr, 10);
  std::vector<std::vector<uint8_t>> seeds;
  for (int i = 3; i < argc; ++i) {
    seeds.push_back(read_file(argv[i]));
    if (seeds.back().empty()) {
      fprintf(stderr, "cannot read %s\n", argv[i]);
      return 2;
    }
  }
  long loaded = 0, rejected = 0;
  pask_geom geom;
  memset(&geom, 0, sizeof(geom));
  for (long r = 0; r < rounds; ++r) {
    std::vector<uint8_t> b = seeds[below((uint32_t)seeds.size())];
    const bool pristine = below(16) == 0;
    if (!pristine) mutate(b);
    uint8_t* heap = static_cast<uint8_t*>(malloc(b.size() ? b.size() : 1));   // exactly sized
    if (!b.empty()) memcpy(heap, b.data(), b.size());
    pask_policy p;
    memset(&p, 0xCD, sizeof(p));
    const pask_geom* gp = nullptr;
    if (below(2)) {
      geom = random_geom();
      gp = &geom;
    }
    const int st = pask_policy_load(heap, b.size(), gp, &p);
    free(heap);
    if (st == PASK_OK) {
      ++loaded;
      if (!table_ok(p)) {
        fprintf(stderr, "round %ld: a blob loaded with an invalid table\n", r);
        return 1;
      }
    } else {
      ++rejected;
      if (st != PASK_E_POLICY && st != PASK_E_SHAPE && st != PASK_E_ARG) {
        fprintf(stderr, "round %ld: unexpected status %d\n", r, st);
        return 1;
      }
    }
    if (pristine && gp == nullptr && st != PASK_OK) {
      fprintf(stderr, "round %ld: a seed blob was rejected (%d)\n", r, st);
      return 1;
    }
    // geometry validation: host-only arithmetic
    pask_geom g = random_geom();
    pask_cache_layout L;
    const int ls = pask_cache_layout_query(&g, &L);
    const size_t nb = pask_cache_bytes(&g);
    if ((ls == PASK_OK) != (nb != 0) || (ls == PASK_OK && (L.total_bytes != nb || L.lo_pool_off < L.hi_pool_off))) {
      fprintf(stderr, "round %ld: layout and size disagree\n", r);
      return 1;
    }
    static const int32_t scal[] = {0, 1, 2, 63, 64, 65, 4096, 65535, 1 << 28, 0x7FFFFFFF, 0x7FFFFF80, -1,
                                   (int32_t)0x80000000};
    const int32_t wb = below(2) ? scal[below(sizeof(scal) / sizeof(scal[0]))] : (int32_t)next_u64();
    const int32_t wh = below(2) ? scal[below(sizeof(scal) / sizeof(scal[0]))] : (int32_t)next_u64();
    pask_geom vg = {64, 36, 32, 8, 128, 16, 9216, 1000, 1000, 0};   // a valid geometry, random batch / hint
    if (below(2)) g = vg;
    const size_t ws = pask_workspace_bytes(&g, wb, wh);
    if ((pask_cache_bytes(&g) != 0) && wb >= 1 && wb <= g.max_batch && ws == 0) {
      fprintf(stderr, "round %ld: no workspace size for a valid geometry\n", r);
      return 1;
    }
  }
  printf("ok: %ld rounds, %ld loaded, %ld rejected\n", rounds, loaded, rejected);
  return loaded > 0 && rejected > 0 ? 0 : 1;
}
