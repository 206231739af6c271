// Host-only harness for the C ABI's validation layer (csrc/abi.hip), built under AddressSanitizer
// and UndefinedBehaviorSanitizer by tests/test_abi_sanitized.py. The kernel launchers are
// replaced by stubs that record their arguments, so no GPU is touched: every entry point is
// called with valid and invalid arguments, and the harness checks the status codes, that
// invalid calls launch nothing, and that the arguments handed to the launchers (derived sizes,
// workspace carve-up) are the documented ones.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <cmath>
#include <limits>
#include <string>
#include <thread>

#include "../../include/dblast.h"
#include "../../paper_2608_05448_amd/csrc/kernels.hpp"

namespace {
int g_launches = 0;
hipError_t g_result = hipSuccess;
dbl::HeadArgs g_head;
dbl::SampleArgs g_sample;
dbl::VerifyArgs g_verify;
dbl::GreedyArgs g_greedy;
int g_fail = 0;

void check(bool ok, const char* what, int line) {
  if (!ok) {
    ++g_fail;
    fprintf(stderr, "FAILED line %d: %s (last error: %s)\n", line, what, dbl_last_error());
  }
}
#define CHECK(x) check((x), #x, __LINE__)

void* P(uintptr_t a) { return reinterpret_cast<void*>(a); }
float* F(uintptr_t a) { return reinterpret_cast<float*>(a); }
int32_t* I(uintptr_t a) { return reinterpret_cast<int32_t*>(a); }
bool inside(const void* p, const void* base, size_t n) {
  const uintptr_t q = reinterpret_cast<uintptr_t>(p), b = reinterpret_cast<uintptr_t>(base);
  return q >= b && q < b + n;
}
}  // namespace

namespace dbl {
hipError_t launch_head(const HeadArgs& a, hipStream_t) { ++g_launches; g_head = a; return g_result; }
hipError_t launch_sample(const SampleArgs& a, hipStream_t) { ++g_launches; g_sample = a; return g_result; }
hipError_t launch_verify(const VerifyArgs& a, hipStream_t) { ++g_launches; g_verify = a; return g_result; }
hipError_t launch_sample_greedy(const GreedyArgs& a, hipStream_t) { ++g_launches; g_greedy = a; return g_result; }
hipError_t launch_verify_greedy(const GreedyArgs& a, hipStream_t) { ++g_launches; g_greedy = a; return g_result; }
hipError_t launch_objective(const ObjectiveArgs&, hipStream_t) { ++g_launches; return g_result; }
hipError_t launch_expand(const ExpandArgs&, hipStream_t) { ++g_launches; return g_result; }
hipError_t launch_prior_head(const PriorHeadArgs&, hipStream_t) { ++g_launches; return g_result; }
hipError_t launch_filter(const FilterArgs&, hipStream_t) { ++g_launches; return g_result; }
hipError_t launch_determinism(const DeterminismArgs&, hipStream_t) { ++g_launches; return g_result; }
hipError_t launch_read_probe(const void*, int64_t, float*, int64_t, hipStream_t) { ++g_launches; return g_result; }
}  // namespace dbl

int main(int argc, char** argv) {
  if (argc > 1 && strcmp(argv[1], "--plant-overflow") == 0) {
    // Shows that the sanitizer is active: one read past a heap array.
    volatile int* v = new int[4];
    const int x = v[argc + 2];
    delete[] v;
    return x == 12345 ? 3 : 2;
  }
  const uintptr_t A = 0x10000;            // fake, aligned device addresses (never dereferenced)
  auto a = [&](int i) { return A + 0x100000 * static_cast<uintptr_t>(i); };
  void* null = nullptr;

  // --- head -------------------------------------------------------------------------------
  dbl_shape hs{2, 4, 3, 64, 1000};
  CHECK(dbl_head_logprobs(hs, DBL_BF16, P(a(0)), P(a(1)), F(a(2)), F(a(3)), F(a(4)), nullptr,
                          null, 0, null) == DBL_OK);
  CHECK(g_launches == 1 && g_head.M == 24 && g_head.V == 1000 && g_head.d == 64 &&
        g_head.dtype_bf16 && g_head.argmax == nullptr && g_head.amax_keys == nullptr);
  const size_t hws = dbl_workspace_bytes(DBL_OP_HEAD, hs);
  CHECK(hws == 256);
  CHECK(dbl_head_logprobs(hs, DBL_F32, P(a(0)), P(a(1)), F(a(2)), F(a(3)), F(a(4)), I(a(5)),
                          P(a(6)), hws, null) == DBL_OK);
  CHECK(g_launches == 2 && g_head.amax_keys == P(a(6)) && !g_head.dtype_bf16);
  int before = g_launches;
  CHECK(dbl_head_logprobs(hs, DBL_BF16, P(a(0) + 8), P(a(1)), F(a(2)), F(a(3)), F(a(4)),
                          nullptr, null, 0, null) == DBL_EINVAL);
  CHECK(dbl_head_logprobs(dbl_shape{2, 4, 3, 60, 1000}, DBL_BF16, P(a(0)), P(a(1)), F(a(2)),
                          F(a(3)), F(a(4)), nullptr, null, 0, null) == DBL_ESHAPE);
  CHECK(dbl_head_logprobs(dbl_shape{1, 1, 1, (1 << 20) + 8, 8}, DBL_BF16, P(a(0)), P(a(1)),
                          F(a(2)), F(a(3)), F(a(4)), nullptr, null, 0, null) == DBL_ESHAPE);
  CHECK(dbl_head_logprobs(dbl_shape{1, 1, 1, 64, 1 << 24}, DBL_BF16, P(a(0)), P(a(1)), F(a(2)),
                          F(a(3)), F(a(4)), nullptr, null, 0, null) == DBL_ESHAPE);
  CHECK(dbl_head_logprobs(dbl_shape{INT64_MAX / 2, 1 << 20, 64, 64, 1 << 23}, DBL_BF16, P(a(0)),
                          P(a(1)), F(a(2)), F(a(3)), F(a(4)), nullptr, null, 0,
                          null) == DBL_ESHAPE);
  CHECK(dbl_head_logprobs(hs, 9, P(a(0)), P(a(1)), F(a(2)), F(a(3)), F(a(4)), nullptr, null, 0,
                          null) == DBL_EDTYPE);
  CHECK(dbl_head_logprobs(hs, DBL_F32, P(a(0)), P(a(1)), F(a(2)), F(a(3)), F(a(4)), I(a(5)),
                          P(a(6)), hws - 1, null) == DBL_EWORKSPACE);
  CHECK(dbl_head_logprobs(hs, DBL_F32, P(a(0)), P(a(1)), F(a(2)), F(a(3)), F(a(4)), I(a(5)),
                          P(a(6) + 16), hws, null) == DBL_EWORKSPACE);
  CHECK(g_launches == before);
  // launch failure -> DBL_EHIP with a message
  g_result = hipErrorInvalidConfiguration;
  CHECK(dbl_head_logprobs(hs, DBL_BF16, P(a(0)), P(a(1)), F(a(2)), F(a(3)), F(a(4)), nullptr,
                          null, 0, null) == DBL_EHIP);
  CHECK(strstr(dbl_last_error(), "DBL_EHIP") != nullptr);
  g_result = hipSuccess;

  // --- sample / verify / expected length: the workspace carve-up ---------------------------
  dbl_shape bs{5, 7, 3, 0, 151936};
  CHECK(dbl_workspace_bytes(DBL_OP_SAMPLE, bs) == 0);
  CHECK(dbl_sample_block(bs, F(a(0)), F(a(1)), F(a(2)), F(a(3)), 0.7f, 9, 2, 11, I(a(4)),
                         I(a(5)), nullptr, 0, null) == DBL_OK);
  CHECK(g_sample.blk.nT == 1187 && g_sample.blk.seq_offset == 11 && g_sample.blk.step == 2 &&
        g_sample.z_out == I(a(4)) && g_sample.x_out == I(a(5)));
  const size_t vws = dbl_workspace_bytes(DBL_OP_VERIFY, bs);
  CHECK(dbl_verify_block(bs, F(a(0)), F(a(1)), F(a(2)), F(a(3)), 1.0f, I(a(4)), F(a(5)), 8, 1,
                         0, 0, I(a(6)), I(a(7)), F(a(8)), nullptr, F(a(9)), P(a(10)), vws,
                         null) == DBL_OK);
  {
    const void* parts[4] = {g_verify.wpost, g_verify.beta_part, g_verify.res_tiles,
                            g_verify.p_tiles};
    for (const void* q : parts)
      CHECK(inside(q, P(a(10)), vws) && reinterpret_cast<uintptr_t>(q) % 256 == 0);
    CHECK(reinterpret_cast<const char*>(g_verify.beta_part) -
              reinterpret_cast<const char*>(g_verify.wpost) >= 5 * 7 * 3 * 8);
    CHECK(g_verify.Kp == 8 && !g_verify.trajectory && g_verify.al == nullptr);
  }
  before = g_launches;
  CHECK(dbl_verify_block(bs, F(a(0)), F(a(1)), F(a(2)), F(a(3)), 1.0f, I(a(4)), F(a(5)), 9, 1,
                         0, 0, I(a(6)), I(a(7)), nullptr, nullptr, nullptr, P(a(10)), vws,
                         null) == DBL_EINVAL);
  CHECK(dbl_verify_block(bs, F(a(0)), F(a(1)), F(a(2)), F(a(3)), 1.0f, I(a(4)), F(a(5)), 8, 1,
                         0, 0, I(a(6)), I(a(7)), nullptr, F(a(8) + 4), nullptr, P(a(10)), vws,
                         null) == DBL_EINVAL);
  CHECK(dbl_verify_block(bs, F(a(0)), F(a(1)), F(a(2)), F(a(3)), -1.0f, I(a(4)), F(a(5)), 8,
                         1, 0, 0, I(a(6)), I(a(7)), nullptr, nullptr, nullptr, P(a(10)), vws,
                         null) == DBL_EINVAL);
  CHECK(dbl_verify_block(bs, F(a(0)), F(a(1)), F(a(2)), F(a(3)), std::nanf(""), I(a(4)),
                         F(a(5)), 8, 1, 0, 0, I(a(6)), I(a(7)), nullptr, nullptr, nullptr,
                         P(a(10)), vws, null) == DBL_EINVAL);
  CHECK(dbl_expected_len(bs, F(a(0)), F(a(1)), F(a(2)), F(a(3)), 1.0f, I(a(4)), F(a(5)),
                         nullptr, F(a(6)), P(a(10)),
                         dbl_workspace_bytes(DBL_OP_EXPECTED_LEN, bs) - 1, null) ==
        DBL_EWORKSPACE);
  CHECK(dbl_sample_block(dbl_shape{1, 1, 65, 0, 100}, F(a(0)), F(a(1)), F(a(2)), F(a(3)), 1.0f,
                         0, 0, 0, I(a(4)), I(a(5)), P(a(6)), 1 << 20, null) == DBL_ESHAPE);
  CHECK(g_launches == before);
  CHECK(dbl_expected_len(bs, F(a(0)), F(a(1)), F(a(2)), F(a(3)), 1.0f, I(a(4)), F(a(5)),
                         nullptr, F(a(6)), P(a(10)), dbl_workspace_bytes(DBL_OP_EXPECTED_LEN, bs),
                         null) == DBL_OK);
  CHECK(g_verify.trajectory && g_verify.res_tiles == nullptr && g_verify.Kp == 7);
  // empty batch: validated, nothing launched
  before = g_launches;
  CHECK(dbl_verify_block(dbl_shape{0, 7, 3, 0, 100}, F(a(0)), F(a(1)), F(a(2)), F(a(3)), 1.0f,
                         I(a(4)), F(a(5)), 7, 0, 0, 0, I(a(6)), I(a(7)), nullptr, nullptr,
                         nullptr, nullptr, 0, null) == DBL_OK);
  CHECK(g_launches == before);

  // --- the allocation-free verification: rejections happen before any runtime call ---------
  before = g_launches;
  {
    dbl_shape big{1024, 16, 8, 0, 151936};  // needs ~19 MiB of scratch
    CHECK(dbl_workspace_bytes(DBL_OP_VERIFY, big) > (size_t(8) << 20));
    CHECK(dbl_verify_block_static(big, F(a(0)), F(a(1)), F(a(2)), F(a(3)), 1.0f, I(a(4)),
                                  F(a(5)), 16, 0, 0, 0, I(a(6)), I(a(7)), nullptr, nullptr,
                                  nullptr, null) == DBL_EWORKSPACE);
    CHECK(strstr(dbl_last_error(), "fixed scratch") != nullptr);
    CHECK(dbl_verify_block_static(bs, F(a(0)), F(a(1)), F(a(2)), F(a(3)), 1.0f, I(a(4)),
                                  F(a(5)) + 1, 7, 0, 0, 0, I(a(6)), I(a(7)), nullptr, nullptr,
                                  nullptr, null) == DBL_EINVAL);
    CHECK(dbl_verify_block_static(bs, F(a(0)), F(a(1)), F(a(2)), F(a(3)), 1.0f, I(a(4)),
                                  F(a(5)), 6, 0, 0, 0, I(a(6)), I(a(7)), nullptr, nullptr,
                                  nullptr, null) == DBL_EINVAL);
    CHECK(dbl_verify_block_static(dbl_shape{0, 7, 3, 0, 100}, F(a(0)), F(a(1)), F(a(2)),
                                  F(a(3)), 1.0f, I(a(4)), F(a(5)), 7, 0, 0, 0, I(a(6)), I(a(7)),
                                  nullptr, nullptr, nullptr, null) == DBL_OK);
  }
  CHECK(g_launches == before);

  // --- greedy ------------------------------------------------------------------------------
  CHECK(dbl_sample_greedy(bs, I(a(0)), F(a(1)), 0.0f, 1, 2, 3, I(a(2)), I(a(3)), null) ==
        DBL_OK);
  CHECK(g_greedy.xhat == I(a(0)) && g_greedy.blk.z_temp == 0.0f);
  const size_t gws = dbl_workspace_bytes(DBL_OP_VERIFY_GREEDY, bs);
  CHECK(dbl_verify_greedy(bs, I(a(0)), F(a(1)), 1.0f, I(a(2)), F(a(3)), 7, 0, 0, 0, I(a(4)),
                          I(a(5)), nullptr, nullptr, nullptr, P(a(6)), gws, null) == DBL_OK);
  CHECK(inside(g_greedy.res_tiles, P(a(6)), gws) && inside(g_greedy.p_tiles, P(a(6)), gws));
  CHECK(dbl_verify_greedy(bs, I(a(0)) + 1, F(a(1)), 1.0f, I(a(2)), F(a(3)), 7, 0, 0, 0, I(a(4)),
                          I(a(5)), nullptr, nullptr, nullptr, P(a(6)), gws, null) == DBL_EINVAL);

  // --- objective, expander, prior head, target, determinism, probe ---------------------------
  CHECK(dbl_acceptance_objective(bs, F(a(0)), F(a(1)), F(a(2)), F(a(3)), 1.0f, I(a(4)),
                                 F(a(5)), 0.1f, nullptr, nullptr, I(a(6)), F(a(7)), F(a(8)),
                                 null) == DBL_OK);
  CHECK(dbl_acceptance_objective(bs, F(a(0)), F(a(1)), F(a(2)), F(a(3)), 1.0f, I(a(4)),
                                 F(a(5)), std::numeric_limits<float>::infinity(), nullptr,
                                 nullptr, I(a(6)), F(a(7)), F(a(8)), null) == DBL_EINVAL);
  CHECK(dbl_expand_branches(dbl_shape{2, 3, 4, 128, 1}, P(a(0)), P(a(1)), P(a(2)), P(a(3)),
                            null) == DBL_OK);
  CHECK(dbl_expand_branches(dbl_shape{2, 3, 4, 100, 1}, P(a(0)), P(a(1)), P(a(2)), P(a(3)),
                            null) == DBL_ESHAPE);
  CHECK(dbl_prior_head(dbl_shape{2, 1, 4, 128, 1}, P(a(0)), P(a(1)), P(a(2)), F(a(3)), null) ==
        DBL_OK);
  CHECK(dbl_target_logprobs(4, 1000, F(a(0)), 1.0f, 20, 0.9f, F(a(1)), nullptr, 0, null) ==
        DBL_OK);
  CHECK(dbl_target_logprobs(4, 1000, F(a(0)), 1.0f, 20, 0.9f, F(a(0)) + 1000, nullptr, 0,
                            null) == DBL_EINVAL);
  CHECK(dbl_early_determinism(3, 4, 100, I(a(0)), F(a(1)), F(a(2)), nullptr, null) == DBL_OK);
  CHECK(dbl_stream_read_probe(P(a(0)), 1 << 20, F(a(1)), 64, null) == DBL_OK);
  CHECK(dbl_stream_read_probe(P(a(0)), (1 << 20) + 4, F(a(1)), 64, null) == DBL_ESHAPE);

  // --- sizes and strings -------------------------------------------------------------------
  CHECK(dbl_workspace_bytes(99, hs) == SIZE_MAX);
  CHECK(dbl_workspace_bytes(DBL_OP_VERIFY, dbl_shape{1, 1, 1, 0, 0}) == SIZE_MAX);
  CHECK(dbl_ntiles(151936) == 1187 && dbl_ntiles(-5) == 0 && dbl_vtile() == 128);
  for (int s = -1; s < 8; ++s) CHECK(dbl_status_string(s) != nullptr);
  // the error text is per thread
  CHECK(dbl_head_logprobs(hs, 9, P(a(0)), P(a(1)), F(a(2)), F(a(3)), F(a(4)), nullptr, null, 0,
                          null) == DBL_EDTYPE);
  std::string other = "unset";
  std::thread t([&] { other = dbl_last_error(); });
  t.join();
  CHECK(other.empty());
  CHECK(std::string(dbl_last_error()).find("DBL_EDTYPE") == 0);

  if (g_fail) {
    fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  printf("abi harness: all checks passed (%d launches recorded)\n", g_launches);
  return 0;
}
