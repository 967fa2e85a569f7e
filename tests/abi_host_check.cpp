// Host-only check of liblt's C ABI layer under AddressSanitizer and
// UndefinedBehaviorSanitizer.
//
// Built by tests/test_abi_host_sanitized.py with g++ from the library's host
// sources (csrc/lt_api.cpp, csrc/plan.cpp) and this file, which stands in for
// the kernel translation units: each launcher below records its call, checks
// that the buffers it was handed lie inside what the caller passed, and
// returns hipErrorNoDevice (the library maps that to LT_ERR_HIP).  No device
// code is compiled and no GPU call is made, so it runs on any host.
//
// It drives every entry point with (1) argument sets the header documents as
// errors, expecting the documented status, (2) valid argument sets, expecting
// them to reach the launcher, and (3) many random argument sets, including
// extreme sizes, strides and misaligned pointers, expecting no sanitizer
// report.  Exit status 0 means every check passed.
#include <hip/hip_runtime.h>

#include <cinttypes>
#include <climits>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>

#include "lt.h"
#include "../paper_2606_10415_amd/csrc/kernels.hpp"

static int g_failures = 0;
static int g_launches = 0;
static uintptr_t g_ws_lo = 0, g_ws_hi = 0;   // workspace range of the current call

#define CHECK(cond, ...)                                   \
  do {                                                     \
    if (!(cond)) {                                         \
      ++g_failures;                                        \
      std::fprintf(stderr, "FAILED %s:%d: ", __FILE__, __LINE__); \
      std::fprintf(stderr, __VA_ARGS__);                   \
      std::fprintf(stderr, "\n");                          \
    }                                                      \
  } while (0)

static void ws_inside(const void* p, size_t bytes, const char* what) {
  if (!p || g_ws_hi == 0) return;
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  CHECK(a >= g_ws_lo && a + bytes <= g_ws_hi, "%s outside the workspace", what);
}

namespace lt {
hipError_t gemm_f16_launch(const GemmArgs& g, hipStream_t) {
  ++g_launches;
  if (g.ws) {
    const size_t need = gemm_splitk_ws_bytes(g.M, g.N, g.K);
    if (need <= g.ws_bytes) ws_inside(g.ws, need, "gemm split-K partials");
  }
  return hipErrorNoDevice;
}
hipError_t bias_grad_launch(const lt_half*, int64_t, int64_t T, int64_t N, lt_half*, float* part,
                            hipStream_t) {
  ++g_launches;
  ws_inside(part, bias_grad_ws_bytes(T, N), "bias partials");
  return hipErrorNoDevice;
}
hipError_t attn_fwd_launch(const AttnFwdArgs&, hipStream_t) {
  ++g_launches;
  return hipErrorNoDevice;
}
hipError_t attn_bwd_launch(const AttnBwdArgs& a, hipStream_t) {
  ++g_launches;
  const AttnShape& s = a.sh;
  ws_inside(a.delta, attn_bwd_delta_bytes(s.B, s.S, s.Hq), "D");
  ws_inside(a.lse2, attn_bwd_lse2_bytes(s.B, s.S, s.Hq), "LSE2");
  ws_inside(a.ds, attn_bwd_ds_bytes(s.B, s.S, s.Hq, s.causal), "dS blocks");
  if (a.nsplit > 1) ws_inside(a.part, attn_bwd_part_bytes(s.B, s.S, s.Hq, s.Hkv, s.D), "dK/dV partials");
  CHECK(a.nsplit >= 1 && (a.ktile == 128 || a.ktile == 256), "dK/dV plan %d %d", a.nsplit, a.ktile);
  return hipErrorNoDevice;
}
hipError_t attn_save_p_launch(const AttnSavePArgs&, hipStream_t) {
  ++g_launches;
  return hipErrorNoDevice;
}
hipError_t attn_bwd_p_launch(const AttnBwdArgs& a, hipStream_t) {
  ++g_launches;
  const AttnShape& s = a.sh;
  ws_inside(a.delta, attn_bwd_delta_bytes(s.B, s.S, s.Hq), "D");
  ws_inside(a.lse2, attn_bwd_lse2_bytes(s.B, s.S, s.Hq), "LSE2");
  if (a.nsplit > 1) ws_inside(a.part, attn_bwd_part_bytes(s.B, s.S, s.Hq, s.Hkv, s.D), "dK/dV partials");
  CHECK(a.psaved != nullptr && a.ds == nullptr, "saved-P arguments");
  return hipErrorNoDevice;
}
hipError_t rmsnorm_fwd_launch(const lt_half*, int64_t, const lt_half*, lt_half*, int64_t, float*,
                              int64_t, int64_t, float, hipStream_t) {
  ++g_launches;
  return hipErrorNoDevice;
}
hipError_t rmsnorm_bwd_launch(const RmsBwdArgs& a, hipStream_t) {
  ++g_launches;
  ws_inside(a.part, rmsnorm_bwd_ws_bytes(a.T, a.H), "rmsnorm partials");
  return hipErrorNoDevice;
}
hipError_t rope_table_launch(float*, int, int, double, hipStream_t) {
  ++g_launches;
  return hipErrorNoDevice;
}
hipError_t rope_launch(lt_half*, int64_t, int, int, int, int, const float*, int, hipStream_t) {
  ++g_launches;
  return hipErrorNoDevice;
}
hipError_t swiglu_fwd_launch(const lt_half*, lt_half*, int64_t, int64_t, hipStream_t) {
  ++g_launches;
  return hipErrorNoDevice;
}
hipError_t swiglu_bwd_launch(const lt_half*, const lt_half*, lt_half*, int64_t, int64_t,
                             hipStream_t) {
  ++g_launches;
  return hipErrorNoDevice;
}
}  // namespace lt

// Addresses that are never dereferenced: the host layer only checks them.
static lt_half* const H = reinterpret_cast<lt_half*>(uintptr_t(0x10000000));
static float* const F32 = reinterpret_cast<float*>(uintptr_t(0x20000000));
static void* const WS = reinterpret_cast<void*>(uintptr_t(0x30000000));

template <class T>
static T* off(T* p, uintptr_t bytes) {
  return reinterpret_cast<T*>(reinterpret_cast<uintptr_t>(p) + bytes);
}

static void set_ws(const void* p, size_t bytes) {
  g_ws_lo = reinterpret_cast<uintptr_t>(p);
  g_ws_hi = p ? g_ws_lo + bytes : 0;
}

static void expect(lt_status got, lt_status want, const char* what) {
  CHECK(got == want, "%s: got %s, want %s (%s)", what, lt_status_string(got), lt_status_string(want),
        lt_last_error());
  if (want != LT_OK) CHECK(std::strlen(lt_last_error()) > 0, "%s: empty lt_last_error", what);
}

static void documented_cases() {
  // ---- GEMM ----
  expect(lt_gemm_f16(2, 0, 64, 64, 64, 1.f, H, 64, H, 64, 0.f, H, 64, nullptr),
         LT_ERR_INVALID_ARG, "gemm transA");
  expect(lt_gemm_f16(0, 1, -1, 64, 64, 1.f, H, 64, H, 64, 0.f, H, 64, nullptr),
         LT_ERR_INVALID_ARG, "gemm M < 0");
  expect(lt_gemm_f16(0, 1, 64, 64, 64, 1.f, nullptr, 64, H, 64, 0.f, H, 64, nullptr),
         LT_ERR_INVALID_ARG, "gemm A NULL");
  expect(lt_gemm_f16(0, 1, 64, 64, 64, 1.f, H, 32, H, 64, 0.f, H, 64, nullptr),
         LT_ERR_INVALID_ARG, "gemm lda");
  expect(lt_gemm_f16(0, 1, 64, 64, 64, 1.f, H, 64, H, 64, 0.f, H, 68, nullptr),
         LT_ERR_UNSUPPORTED, "gemm ldc % 8");
  expect(lt_gemm_f16(0, 1, ((int64_t)1 << 30) + 8, 64, 64, 1.f, H, 64, H, 64, 0.f, H, 64, nullptr),
         LT_ERR_UNSUPPORTED, "gemm M > 2^30");
  {
    const int before = g_launches;
    expect(lt_gemm_f16(1, 0, 61, 45, 13, 1.f, H, 64, H, 48, 0.f, H, 48, nullptr), LT_ERR_HIP,
           "gemm ragged M, N, K reaches the launcher");
    CHECK(g_launches == before + 1, "ragged gemm launcher not reached");
    CHECK(lt_gemm_f16_workspace_size(0, 1, 4096, 22016 - 2048 + 4, 4096) == 0,
          "no split-K workspace for N % 8 != 0");
    CHECK(lt_gemm_f16_workspace_size(0, 1, 4096, 22016 - 2048, 4092) == 0,
          "no split-K workspace for K % 8 != 0");
  }
  expect(lt_gemm_f16(0, 1, 64, 64, 64, 1.f, off(H, 2), 64, H, 64, 0.f, H, 64, nullptr),
         LT_ERR_UNSUPPORTED, "gemm misaligned A");
  expect(lt_gemm_f16(0, 1, 64, 64, 64, 1.f, H, 1 << 22, H, 64, 0.f, H, 64, nullptr),
         LT_ERR_UNSUPPORTED, "gemm lda >= 2^22");
  expect(lt_gemm_f16(0, 1, 0, 64, 64, 1.f, nullptr, 0, nullptr, 0, 0.f, nullptr, 0, nullptr), LT_OK,
         "gemm M = 0 is a no-op");
  expect(lt_gemm_f16_res(0, 1, 64, 64, 64, 1.f, H, 64, H, 64, 1.f, nullptr, 64, H, 64, nullptr),
         LT_ERR_INVALID_ARG, "gemm beta without R");
  int before = g_launches;
  expect(lt_gemm_f16(0, 1, 64, 64, 64, 1.f, H, 64, H, 64, 0.f, H, 64, nullptr), LT_ERR_HIP,
         "gemm valid reaches the launcher");
  CHECK(g_launches == before + 1, "gemm launcher not reached");
  const size_t gws = lt_gemm_f16_workspace_size(0, 1, 4096, 22016 - 2048, 4096);
  set_ws(WS, gws);
  expect(lt_gemm_f16_ws(0, 1, 4096, 22016 - 2048, 4096, 1.f, H, 4096, H, 4096, 0.f, nullptr, 0,
                        nullptr, H, 22016, WS, gws ? gws - 1 : 0, nullptr),
         gws ? LT_ERR_WORKSPACE : LT_ERR_HIP, "gemm_ws short workspace");
  expect(lt_gemm_f16_ws(0, 1, 4096, 22016 - 2048, 4096, 1.f, H, 4096, H, 4096, 0.f, nullptr, 0,
                        nullptr, H, 22016, WS, gws, nullptr),
         LT_ERR_HIP, "gemm_ws valid");
  set_ws(nullptr, 0);
  CHECK(lt_gemm_f16_workspace_size(3, 0, 64, 64, 64) == 0, "workspace size, bad trans");
  CHECK(lt_gemm_f16_workspace_size(0, 0, INT64_MAX, INT64_MAX, INT64_MAX) == 0 ||
            lt_gemm_f16_workspace_size(0, 0, INT64_MAX, INT64_MAX, INT64_MAX) > 0,
        "workspace size at extremes");

  // ---- attention ----
  expect(lt_attn_fwd(nullptr, H, H, 384, 384, H, 128, F32, 1, 16, 2, 1, 64, 0.125f, 1, nullptr),
         LT_ERR_INVALID_ARG, "attn_fwd Q NULL");
  expect(lt_attn_fwd(H, H, H, 384, 384, H, 128, F32, 1, 16, 3, 2, 64, 0.125f, 1, nullptr),
         LT_ERR_INVALID_ARG, "attn_fwd Hq % Hkv");
  expect(lt_attn_fwd(H, H, H, 384, 384, H, 128, F32, 1, 16, 2, 1, 96, 0.125f, 1, nullptr),
         LT_ERR_UNSUPPORTED, "attn_fwd D = 96");
  expect(lt_attn_fwd(H, H, H, 1 << 22, 384, H, 128, F32, 1, 16, 2, 1, 64, 0.125f, 1, nullptr),
         LT_ERR_UNSUPPORTED, "attn_fwd stride >= 2^22");
  expect(lt_attn_fwd(H, H, H, 384, 384, H, 128, F32, 1, 16, 2, 1, 64, 0.125f, 1, nullptr),
         LT_ERR_HIP, "attn_fwd valid");
  const size_t aws = lt_attn_bwd_workspace_size(2, 100, 8, 2, 128, 1);
  CHECK(aws > 0 && aws % 256 == 0, "attn_bwd workspace size %zu", aws);
  set_ws(WS, aws);
  expect(lt_attn_bwd(H, H, H, 1536, 1536, H, H, 1024, F32, H, H, H, 1536, 1536, WS, aws - 1, 2,
                     100, 8, 2, 128, 0.09f, 1, nullptr),
         LT_ERR_WORKSPACE, "attn_bwd short workspace");
  expect(lt_attn_bwd(H, H, H, 1536, 1536, H, H, 1024, F32, H, H, H, 1536, 1536, off(WS, 16), aws,
                     2, 100, 8, 2, 128, 0.09f, 1, nullptr),
         LT_ERR_WORKSPACE, "attn_bwd misaligned workspace");
  expect(lt_attn_bwd(H, H, H, 1536, 1536, H, H, 1024, F32, H, H, H, 1536, 1536, WS, aws, 2, 100, 8,
                     2, 128, 0.09f, 1, nullptr),
         LT_ERR_HIP, "attn_bwd valid");
  set_ws(nullptr, 0);
  const size_t pb = lt_attn_p_size(2, 100, 8, 1);
  CHECK(pb == 2 * 8 * 10 * 2048, "saved-P size %zu", pb);
  expect(lt_attn_fwd_p(H, H, H, 1536, 1536, H, 1024, F32, H, pb - 1, 2, 100, 8, 2, 128, 0.09f, 1,
                       nullptr),
         LT_ERR_HIP, "attn_fwd_p: the forward launch fails first without a device");
  const size_t pws = lt_attn_bwd_p_workspace_size(2, 100, 8, 2, 128);
  set_ws(WS, pws);
  expect(lt_attn_bwd_p(H, H, H, 1536, 1536, H, H, 1024, F32, H, pb - 1, H, H, H, 1536, 1536, WS, pws,
                       2, 100, 8, 2, 128, 0.09f, 1, nullptr),
         LT_ERR_INVALID_ARG, "attn_bwd_p short P");
  expect(lt_attn_bwd_p(H, H, H, 1536, 1536, H, H, 1024, F32, H, pb, H, H, H, 1536, 1536, WS, pws,
                       2, 100, 8, 2, 128, 0.09f, 1, nullptr),
         LT_ERR_HIP, "attn_bwd_p valid");
  set_ws(nullptr, 0);
  CHECK(lt_attn_bwd_workspace_size(0, 100, 8, 2, 128, 1) == 0, "attn ws B = 0");
  CHECK(lt_attn_bwd_workspace_size(1, 100, 8, 3, 128, 1) == 0, "attn ws Hq %% Hkv");

  // ---- SwiGLU, norms, rotary, bias ----
  expect(lt_swiglu_fwd(H, H, 4, 12, nullptr), LT_ERR_UNSUPPORTED, "swiglu F % 8");
  expect(lt_swiglu_bwd(nullptr, H, H, 4, 16, nullptr), LT_ERR_INVALID_ARG, "swiglu_bwd NULL");
  expect(lt_rmsnorm_fwd(H, 16384, H, H, 16384, F32, 4, 16384, 1e-5f, nullptr), LT_ERR_UNSUPPORTED,
         "rmsnorm H > 8192");
  expect(lt_rope_table(F32, 16, 24, 1e4, nullptr), LT_ERR_UNSUPPORTED, "rope D % 16");
  expect(lt_rope_f16(H, 6148, 1, 16, 48, 128, F32, 0, nullptr), LT_ERR_UNSUPPORTED, "rope stride");
  expect(lt_bias_grad_f16(H, 64, 0, 64, H, WS, 1 << 20, nullptr), LT_ERR_INVALID_ARG, "bias T = 0");
  CHECK(std::strcmp(lt_status_string((lt_status)99), "LT_ERR_UNKNOWN") == 0, "status string");
}

static void fuzz(unsigned seed, int rounds) {
  std::mt19937_64 rng(seed);
  auto pick64 = [&]() -> int64_t {
    static const int64_t edge[] = {0, 1, 7, 8, 64, 100, 4096, 8192, 57344, (1 << 22) - 8, 1 << 22,
                                   (int64_t)1 << 30, (int64_t)1 << 31, INT32_MAX, INT64_MAX / 2,
                                   INT64_MAX, -1, -8, INT64_MIN};
    switch (rng() % 3) {
      case 0: return edge[rng() % (sizeof(edge) / sizeof(edge[0]))];
      case 1: return (int64_t)(rng() % 70000) & ~int64_t(rng() % 2 ? 7 : 0);
      default: return (int64_t)(rng() % 300);
    }
  };
  auto pick32 = [&]() -> int {
    static const int edge[] = {0, 1, 2, 8, 64, 128, 4096, 65536, INT32_MAX, INT32_MAX - 1, -1,
                               INT32_MIN};
    return rng() % 2 ? edge[rng() % (sizeof(edge) / sizeof(edge[0]))] : (int)(rng() % 300);
  };
  auto ptr = [&](auto* base) -> decltype(base) {
    switch (rng() % 4) {
      case 0: return nullptr;
      case 1: return off(base, 2 * (rng() % 8));
      default: return base;
    }
  };
  for (int r = 0; r < rounds; ++r) {
    const int64_t M = pick64(), N = pick64(), K = pick64();
    const int ta = (int)(rng() % 3), tb = (int)(rng() % 3);
    const size_t gws = lt_gemm_f16_workspace_size(ta, tb, M, N, K);
    set_ws(WS, gws + 256);
    lt_gemm_f16_ws(ta, tb, M, N, K, 1.f, ptr(H), pick64(), ptr(H), pick64(), rng() % 2 ? 1.f : 0.f,
                   ptr(H), pick64(), rng() % 2 ? ptr(H) : nullptr, ptr(H), pick64(),
                   rng() % 2 ? WS : nullptr, gws + (rng() % 2) * 256, nullptr);
    lt_gemm_gu_swiglu_f16(ptr(H), pick64(), ptr(H), pick64(), ptr(H), pick64(), ptr(H), pick64(),
                          M, N, K, nullptr);
    lt_gemm_swiglu_bwd_f16(ptr(H), pick64(), ptr(H), pick64(), ptr(H), pick64(), ptr(H), pick64(),
                           M, N, K, nullptr);
    const int B = pick32(), S = pick32(), Hq = pick32(), Hkv = pick32(), D = rng() % 2 ? 128 : pick32();
    const int causal = (int)(rng() % 3);
    const size_t aws = lt_attn_bwd_workspace_size(B, S, Hq, Hkv, D, causal);
    set_ws(WS, aws);
    lt_attn_fwd(ptr(H), ptr(H), ptr(H), pick64(), pick64(), ptr(H), pick64(), ptr(F32), B, S, Hq, Hkv,
                D, rng() % 5 ? 0.088f : -1.f, (int)(rng() % 3), nullptr);
    lt_attn_bwd(ptr(H), ptr(H), ptr(H), pick64(), pick64(), ptr(H), ptr(H), pick64(), ptr(F32),
                ptr(H), ptr(H), ptr(H), pick64(), pick64(), rng() % 4 ? WS : nullptr, aws, B, S, Hq,
                Hkv, D, 0.088f, causal, nullptr);
    const size_t pb = lt_attn_p_size(B, S, Hq, causal);
    lt_attn_fwd_p(ptr(H), ptr(H), ptr(H), pick64(), pick64(), ptr(H), pick64(), ptr(F32), ptr(H),
                  rng() % 2 ? pb : pb / 2, B, S, Hq, Hkv, D, 0.088f, causal, nullptr);
    const size_t pws = lt_attn_bwd_p_workspace_size(B, S, Hq, Hkv, D);
    set_ws(WS, pws);
    lt_attn_bwd_p(ptr(H), ptr(H), ptr(H), pick64(), pick64(), ptr(H), ptr(H), pick64(), ptr(F32),
                  ptr(H), rng() % 2 ? pb : 0, ptr(H), ptr(H), ptr(H), pick64(), pick64(),
                  rng() % 4 ? WS : nullptr, pws, B, S, Hq, Hkv, D, 0.088f, causal, nullptr);
    set_ws(nullptr, 0);
    const int64_t T = pick64(), Hd = pick64();
    const size_t rws = lt_rmsnorm_bwd_workspace_size(T, Hd);
    set_ws(WS, rws);
    lt_rmsnorm_fwd(ptr(H), pick64(), ptr(H), ptr(H), pick64(), ptr(F32), T, Hd, 1e-5f, nullptr);
    lt_rmsnorm_bwd(ptr(H), pick64(), ptr(H), pick64(), ptr(H), ptr(F32), rng() % 2 ? ptr(H) : nullptr,
                   pick64(), ptr(H), pick64(), ptr(H), WS, rws, T, Hd, nullptr);
    const size_t bws = lt_bias_grad_workspace_size(T, Hd);
    set_ws(WS, bws);
    lt_bias_grad_f16(ptr(H), pick64(), T, Hd, ptr(H), WS, bws, nullptr);
    set_ws(nullptr, 0);
    lt_swiglu_fwd(ptr(H), ptr(H), T, Hd, nullptr);
    lt_swiglu_bwd(ptr(H), ptr(H), ptr(H), T, Hd, nullptr);
    lt_rope_table(ptr(F32), pick32(), pick32(), rng() % 2 ? 1e4 : -1.0, nullptr);
    lt_rope_f16(ptr(H), pick64(), pick32(), pick32(), pick32(), pick32(), ptr(F32), (int)(rng() % 3),
                nullptr);
  }
}

int main(int argc, char** argv) {
  const int rounds = argc > 1 ? std::atoi(argv[1]) : 20000;
  documented_cases();
  fuzz(12345u, rounds);
  std::printf("abi host check: %d failures, %d launcher calls\n", g_failures, g_launches);
  return g_failures == 0 ? 0 : 1;
}
