// Reuse-phase matcher (Sec. "Reuse"): find where the tail of the generated
// output reappears in the original code, so that the original tokens after
// it become the next draft.  Host code; O(n_orig * max_ngram) per call.

#include <stdint.h>

#include <string>

#include "../../include/ee.h"

extern "C" int32_t ee_match_reuse(const int32_t* generated, int32_t n_gen, const int32_t* original,
                                  int32_t n_orig, int32_t cursor, int32_t min_ngram, int32_t max_ngram,
                                  int32_t* draft_start, int32_t* match_len) {
  if (!draft_start || !match_len) return EE_EINVAL;
  if (n_gen < 0 || n_orig < 0 || min_ngram < 1 || max_ngram < min_ngram) return EE_EINVAL;
  if ((n_gen > 0 && !generated) || (n_orig > 0 && !original)) return EE_EINVAL;
  *draft_start = -1;
  *match_len = 0;
  const int32_t top = max_ngram < n_gen ? max_ngram : n_gen;
  for (int32_t len = top; len >= min_ngram; --len) {
    const int32_t* suf = generated + (n_gen - len);
    // window [j, j + len) must end at or after the cursor and leave a draft
    // (a cursor at or below len puts no bound on j; no overflow for any cursor)
    int32_t j = cursor <= len ? 0 : cursor - len;
    for (; j + len < n_orig; ++j) {
      int32_t i = 0;
      while (i < len && original[j + i] == suf[i]) ++i;
      if (i == len) {
        *draft_start = j + len;
        *match_len = len;
        return EE_OK;
      }
    }
  }
  return EE_OK;
}
