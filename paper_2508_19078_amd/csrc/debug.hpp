// Host-side range checks of the device-resident maps an entry point indexes
// memory through, run only when the environment variable FLUXMOE_DEBUG_CHECKS
// is set (and not "0").  Each check copies the map to the host on the call's
// stream, waits for it, and returns MOE_ERR_ARG naming the first bad entry
// before anything is launched; a check therefore synchronises the stream and
// cannot run under HIP graph capture.  The maps normally come from
// moe_permute, which writes them in range; the checks are for debugging a
// caller that builds or edits them itself.
#pragma once

#include <stdlib.h>

#include <vector>

#include "common.hpp"

namespace fm {

inline bool debug_checks() {
  const char* v = getenv("FLUXMOE_DEBUG_CHECKS");
  return v && v[0] && !(v[0] == '0' && v[1] == '\0');
}

inline int debug_fetch(const int32_t* dev, size_t n, std::vector<int32_t>& out, hipStream_t st, const char* what) {
  out.assign(n, 0);
  if (n > 0 && hipMemcpyAsync(out.data(), dev, n * sizeof(int32_t), hipMemcpyDeviceToHost, st) != hipSuccess)
    return fail(MOE_ERR_HIP, "debug check: copy of %s failed", what);
  if (hipStreamSynchronize(st) != hipSuccess) return fail(MOE_ERR_HIP, "debug check: stream synchronisation failed");
  return MOE_OK;
}

// offsets [S_routed + 1]: 0 first, non-decreasing, at most T * k rows.
inline int debug_check_offsets(const int32_t* offsets, int S_routed, int T, int k, hipStream_t st) {
  std::vector<int32_t> h;
  FM_TRY(debug_fetch(offsets, (size_t)S_routed + 1, h, st, "offsets"));
  if (h[0] != 0) return fail(MOE_ERR_ARG, "debug check: offsets[0]=%d, must be 0", h[0]);
  for (int s = 0; s < S_routed; ++s)
    if (h[s + 1] < h[s]) return fail(MOE_ERR_ARG, "debug check: offsets[%d]=%d < offsets[%d]=%d", s + 1, h[s + 1], s, h[s]);
  if ((long long)h[S_routed] > (long long)T * k)
    return fail(MOE_ERR_ARG, "debug check: offsets[%d]=%d > T*k=%lld", S_routed, h[S_routed], (long long)T * k);
  return MOE_OK;
}

// inv [T, k]: every entry decodes (p, or -2-p for a folded choice) to a routed
// row p in [0, T * k).
inline int debug_check_inv(const int32_t* inv, int T, int k, hipStream_t st) {
  std::vector<int32_t> h;
  FM_TRY(debug_fetch(inv, (size_t)T * k, h, st, "inv"));
  const long long R = (long long)T * k;
  for (size_t i = 0; i < h.size(); ++i) {
    const long long p = h[i] >= 0 ? h[i] : -2LL - h[i];
    if (p < 0 || p >= R)
      return fail(MOE_ERR_ARG, "debug check: inv[%zu]=%d decodes to row %lld outside [0, %lld)", i, h[i], p, R);
  }
  return MOE_OK;
}

// perm_token [rows]: tokens in [0, T).
inline int debug_check_tokens(const int32_t* perm_token, int rows, int T, hipStream_t st) {
  std::vector<int32_t> h;
  FM_TRY(debug_fetch(perm_token, (size_t)rows, h, st, "perm_token"));
  for (int i = 0; i < rows; ++i)
    if (h[i] < 0 || h[i] >= T) return fail(MOE_ERR_ARG, "debug check: perm_token[%d]=%d outside [0, %d)", i, h[i], T);
  return MOE_OK;
}

// The routed rows offsets[S_routed] (after debug_check_offsets).
inline int debug_rows(const int32_t* offsets, int S_routed, hipStream_t st, int* rows) {
  std::vector<int32_t> h;
  FM_TRY(debug_fetch(offsets + S_routed, 1, h, st, "offsets"));
  *rows = h[0];
  return MOE_OK;
}

}  // namespace fm
