// Drives the C-ABI's host paths under AddressSanitizer / UndefinedBehavior-
// Sanitizer (built with g++ against the launch stubs of api_stubs.cpp): plan
// introspection over many shapes and settings, and the argument checks of
// pat_allgather / pat_reducescatter, the remembered pointer set included.
#include <cstdint>
#include <cstdio>
#include <vector>

#include "../../include/pat.h"

static int failures = 0;
#define EXPECT(cond)                                                        \
  do {                                                                      \
    if (!(cond)) {                                                          \
      std::fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                           \
    }                                                                       \
  } while (0)

static std::vector<void*> fake(uintptr_t base, int n, uintptr_t stride) {
  std::vector<void*> v(n);
  for (int i = 0; i < n; ++i) v[i] = (void*)(base + uintptr_t(i) * stride);
  return v;
}

int main() {
  long plans = 0;
  const int ns[] = {1, 2, 3, 5, 6, 7, 8, 9, 13, 16, 24, 33, 64, 100, 127, 128, 129, 1000, 4097};
  const size_t counts[] = {1, 3, 8, 17, 64, 1000, 4104, 262144};
  const size_t budgets[] = {0, 64, 4096, 65536, size_t(8) << 20};
  for (int order = 0; order < 2; ++order)
    for (int fusion = 0; fusion < 3; ++fusion)
      for (size_t b : budgets) {
        EXPECT(pat_set_linear_order(order) == PAT_OK);
        EXPECT(pat_set_top_fusion(fusion) == PAT_OK);
        EXPECT(pat_set_buffer_bytes(b) == PAT_OK);
        for (int n : ns)
          for (size_t c : counts)
            for (int dt = 0; dt < 3; ++dt)
              for (int coll = 0; coll < 2; ++coll) {
                if (n >= 1000 && c > 1000) continue;
                pat_plan_info_t info;
                const pat_status_t s = pat_plan_info((pat_collective_t)coll, n, c, (pat_dtype_t)dt, &info);
                EXPECT(s == PAT_OK);
                if (s != PAT_OK) continue;
                EXPECT(info.fused_steps >= 0 && info.fused_steps <= info.steps);
                EXPECT(info.launches_per_op >= 1 || n == 1);
                int nsteps = 0, nentries = 0;
                pat_plan_steps((pat_collective_t)coll, n, c, (pat_dtype_t)dt, nullptr, nullptr, 0, nullptr, nullptr,
                               nullptr, nullptr, 0, &nsteps, &nentries);
                std::vector<int32_t> d(nsteps), k(nsteps), p(nentries), a(nentries), bb(nentries), cc(nentries);
                EXPECT(pat_plan_steps((pat_collective_t)coll, n, c, (pat_dtype_t)dt, d.data(), k.data(), nsteps,
                                      p.data(), a.data(), bb.data(), cc.data(), nentries, &nsteps,
                                      &nentries) == PAT_OK);
                long edges = 0;
                for (int s2 = 0; s2 < nsteps; ++s2) edges += k[s2];
                EXPECT(edges == n - 1);
                ++plans;
              }
      }
  pat_set_buffer_bytes(0);
  pat_set_top_fusion(0);
  pat_set_linear_order(0);

  // Argument checks.  Valid sets may reach the device layer (no GPU here:
  // PAT_ERR_HIP; with one, the stub launches run nothing); every invalid set
  // must be refused, also right after a valid one was remembered.
  const int n = 64;
  const size_t count = 1000;  // 4000-byte chunks
  auto send = fake(0x10000000, n, 0x100000), recv = fake(0x80000000, n, 0x100000);
  const pat_status_t first = pat_allgather(send.data(), recv.data(), count, PAT_FLOAT32, n, nullptr);
  EXPECT(first != PAT_ERR_INVALID_ARGUMENT);
  EXPECT(pat_allgather(send.data(), recv.data(), count, PAT_FLOAT32, n, nullptr) == first);
  EXPECT(pat_allgather(send.data(), recv.data(), 0x40000, PAT_FLOAT32, n, nullptr) == PAT_ERR_INVALID_ARGUMENT);
  EXPECT(pat_allgather(send.data(), recv.data(), count, PAT_FLOAT32, n, nullptr) == first);
  auto overlap = recv;
  overlap[7] = (char*)overlap[6] + 64;
  EXPECT(pat_allgather(send.data(), overlap.data(), count, PAT_FLOAT32, n, nullptr) == PAT_ERR_INVALID_ARGUMENT);
  auto misaligned = send;
  misaligned[3] = (char*)misaligned[3] + 2;
  EXPECT(pat_allgather(misaligned.data(), recv.data(), count, PAT_FLOAT32, n, nullptr) == PAT_ERR_INVALID_ARGUMENT);
  auto nul = send;
  nul[n - 1] = nullptr;
  EXPECT(pat_reducescatter(nul.data(), recv.data(), count, PAT_FLOAT32, PAT_SUM, n, nullptr) ==
         PAT_ERR_INVALID_ARGUMENT);
  // reduce-scatter: send rows of n * count elements
  auto rs_send = fake(0x100000000, n, 0x1000000), rs_recv = fake(0x300000000, n, 0x10000);
  const pat_status_t rs = pat_reducescatter(rs_send.data(), rs_recv.data(), count, PAT_BFLOAT16, PAT_SUM, n, nullptr);
  EXPECT(rs != PAT_ERR_INVALID_ARGUMENT);
  EXPECT(pat_reducescatter(rs_send.data(), rs_recv.data(), count, PAT_BFLOAT16, PAT_SUM, n, nullptr) == rs);
  EXPECT(pat_reducescatter(rs_send.data(), rs_recv.data(), 0x10000, PAT_BFLOAT16, PAT_SUM, n, nullptr) ==
         PAT_ERR_INVALID_ARGUMENT);
  // the entry point that allocates nothing: the same checks; a valid set
  // stops at the device layer (here: PAT_ERR_HIP), never at the checks
  const pat_status_t na =
      pat_reducescatter_noalloc(rs_send.data(), rs_recv.data(), count, PAT_BFLOAT16, PAT_SUM, n, nullptr);
  EXPECT(na != PAT_ERR_INVALID_ARGUMENT && na != PAT_OK);
  EXPECT(pat_reducescatter_noalloc(rs_send.data(), rs_recv.data(), 0x10000, PAT_BFLOAT16, PAT_SUM, n, nullptr) ==
         PAT_ERR_INVALID_ARGUMENT);
  EXPECT(pat_reducescatter_noalloc(nul.data(), recv.data(), count, PAT_FLOAT32, PAT_SUM, n, nullptr) ==
         PAT_ERR_INVALID_ARGUMENT);
  EXPECT(pat_reducescatter_noalloc(rs_send.data(), rs_recv.data(), count, PAT_FLOAT32, (pat_op_t)3, n, nullptr) ==
         PAT_ERR_UNSUPPORTED);
  EXPECT(pat_reducescatter_noalloc(rs_send.data(), rs_recv.data(), 0, PAT_FLOAT32, PAT_SUM, n, nullptr) == PAT_OK);
  EXPECT(pat_allgather(nullptr, recv.data(), count, PAT_FLOAT32, n, nullptr) == PAT_ERR_INVALID_ARGUMENT);
  EXPECT(pat_allgather(send.data(), recv.data(), count, PAT_FLOAT32, 0, nullptr) == PAT_ERR_INVALID_ARGUMENT);
  pat_finalize();
  std::printf("%ld plans checked, %d failures\n", plans, failures);
  return failures ? 1 : 0;
}
