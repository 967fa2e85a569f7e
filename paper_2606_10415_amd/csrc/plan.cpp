// Host-side launch planning of liblt (no device code): which GEMM launches
// take a split-K last wave and how much workspace that needs.  Compiled into
// the library with the kernels, and on its own into the host-only sanitizer
// check of the C ABI.
#include "kernels.hpp"

namespace lt {

bool gemm_splitk_tail(int64_t M, int64_t N, int64_t K, SplitTail* p) {
  // the geometry of the half-tile tail (256x256 tiles, one wave = 256 CUs),
  // with the last wave's K split so that its units fill about one wave; a
  // launch of less than about one wave of 256x256 tiles is split whole
  // (split_at = 0: no full-K part) when that beats 128x128 tiles with full
  // K: the split gives twice their workgroups (S = 8) or each split still
  // runs a long K loop (K / S >= kLongK); otherwise the workspace round trip
  // costs more than the larger tile saves
  constexpr int64_t kCUs = 256, kMinSlices = 8, kMaxSplits = 8, kLongK = 2048;
  if (M <= 0 || N <= 0 || K <= 0) return false;
  // the partial tiles and their sum move 8 columns at a time, and a ragged K
  // takes its own launch: both need multiples of 8
  if ((N & 7) || (K & 7)) return false;
  // beyond the sizes the GEMM entry points accept: no plan (and no overflow)
  if (M > ((int64_t)1 << 30) || N > ((int64_t)1 << 30) || K > ((int64_t)1 << 30)) return false;
  const int64_t tm = (M + 255) / 256, tn = (N + 255) / 256, tiles = tm * tn;
  const int64_t nk = (K + 63) / 64;
  if (tiles < 192) {
    int64_t S = kCUs / tiles;
    if (S > kMaxSplits) S = kMaxSplits;
    if (S > nk / kMinSlices) S = nk / kMinSlices;
    if (S < 2) return false;
    if (S < kMaxSplits && K < kLongK * S) return false;
    p->columns = true;
    p->split_at = 0;
    p->Mt = M;
    p->Nt = N;
    p->S = (int)S;
    return true;
  }
  const int64_t waves = tiles / kCUs, rem = tiles % kCUs;
  if (waves < 1 || rem == 0 || 2 * rem > kCUs) return false;
  int64_t S = kCUs / rem;
  if (S > kMaxSplits) S = kMaxSplits;
  if (S > nk / kMinSlices) S = nk / kMinSlices;
  if (S < 2) return false;
  const int64_t full = waves * kCUs;
  if (full % tm == 0 && full / tm < tn) {
    p->columns = true;
    p->split_at = (full / tm) * 256;
    p->Mt = M;
    p->Nt = N - p->split_at;
  } else if (full % tn == 0 && full / tn < tm) {
    p->columns = false;
    p->split_at = (full / tn) * 256;
    p->Mt = M - p->split_at;
    p->Nt = N;
  } else {
    return false;
  }
  p->S = (int)S;
  return true;
}

size_t gemm_splitk_ws_bytes(int64_t M, int64_t N, int64_t K) {
  SplitTail p;
  if (!gemm_splitk_tail(M, N, K, &p)) return 0;
  return (size_t)p.S * (size_t)p.Mt * (size_t)p.Nt * sizeof(float);
}

}  // namespace lt
