// Edit-session driver behind ee_edit_begin / ee_edit_step (include/ee.h):
// the Reuse / Generate phase machine of Sec. "Reuse" and Sec. "Generate",
// written on the public C ABI only (verification, extension, rollback and the
// matcher); host control flow, no kernels of its own.

#include <string.h>

#include <algorithm>
#include <vector>

#include "../../include/ee.h"

namespace {

int32_t state_of(ee_ctx* c, int32_t seq, int32_t* len, int32_t* pending) {
  return ee_seq_state(c, seq, len, pending);
}

// Matcher with the session's suffix lengths; while the output is shorter than
// the shortest length, the whole output is matched.
int32_t match(const int32_t* out, int32_t n_out, const int32_t* original, int32_t n_orig, int32_t cursor,
              const ee_edit_params* p, int32_t* ds) {
  const int32_t lo = std::min(p->min_match, n_out), hi = std::max(lo, p->max_match);
  int32_t ml;
  return ee_match_reuse(out, n_out, original, n_orig, cursor, lo, hi, ds, &ml);
}

// Make the draft sequence follow the output: committed = prompt + out[0..j),
// pending = out[j] for the j its length implies; returns the lag m - j (m =
// n_out - 1, the index of the target's pending token).
int32_t align_draft(ee_ctx* target, int32_t seq, ee_ctx* draft, int32_t dseq, const int32_t* out,
                    int32_t n_out, int32_t* lag) {
  int32_t tl, tp, dl, dp, rc;
  if ((rc = state_of(target, seq, &tl, &tp)) || (rc = state_of(draft, dseq, &dl, &dp))) return rc;
  if (dl > tl) {   // an earlier step stopped after the draft ran ahead
    if ((rc = ee_kv_rollback(draft, dseq, tl, tp))) return rc;
    dl = tl;
    dp = tp;
  }
  const int32_t l = tl - dl;
  if (l > n_out - 1 || dp != out[n_out - 1 - l]) return EE_ESTATE;
  *lag = l;
  return EE_OK;
}

}  // namespace

extern "C" {

int32_t ee_edit_begin(ee_ctx* target, int32_t seq, ee_ctx* draft, int32_t dseq, ee_edit_state* st) {
  if (!target || !st) return EE_EINVAL;
  int32_t tl, tp, rc;
  if ((rc = state_of(target, seq, &tl, &tp))) return rc;
  if (tp < 0) return EE_ESTATE;
  if (draft) {
    int32_t dl, dp;
    if ((rc = state_of(draft, dseq, &dl, &dp))) return rc;
    if (dl != tl || dp < 0) return EE_ESTATE;   // both must hold the same prompt
    if ((rc = ee_kv_rollback(draft, dseq, dl, tp))) return rc;
  }
  memset(st, 0, sizeof *st);
  st->phase = EE_PHASE_REUSE;
  st->last_phase = -1;
  return EE_OK;
}

int32_t ee_edit_step(ee_ctx* target, int32_t seq, ee_ctx* draft, int32_t dseq, const int32_t* original,
                     int32_t n_orig, const ee_edit_params* p, ee_edit_state* st, int32_t* out, int32_t n_out,
                     int32_t out_cap, int32_t* n_new) {
  if (!target || !p || !st || !out || !n_new || n_out < 1 || n_orig < 0 || (n_orig > 0 && !original))
    return EE_EINVAL;
  if (p->k_reuse < 1 || p->gamma < 1 || p->top_k < 0 || p->top_k > 8 || p->min_match < 1 ||
      p->max_match < p->min_match)
    return EE_EINVAL;
  if (st->phase != EE_PHASE_REUSE && st->phase != EE_PHASE_GENERATE) return EE_EINVAL;
  if (st->cursor < 0) return EE_EINVAL;   // (the fallback draft starts there: never before original[0])
  if ((int64_t)out_cap < (int64_t)n_out + std::max(p->k_reuse, p->gamma) + 1) return EE_EINVAL;
  int32_t tl, tp, rc;
  if ((rc = state_of(target, seq, &tl, &tp))) return rc;
  if (tp != out[n_out - 1]) return EE_ESTATE;
  *n_new = 0;

  int32_t phase = st->phase;
  int32_t a = 0, nxt = -1;
  std::vector<int32_t> d;
  if (phase == EE_PHASE_REUSE) {
    int32_t ds;
    if ((rc = match(out, n_out, original, n_orig, st->cursor, p, &ds))) return rc;
    const int32_t start = ds >= 0 ? ds : std::min(st->cursor, n_orig);
    const int32_t k = std::min(p->k_reuse, n_orig - start);
    if (k < 1) {
      phase = EE_PHASE_GENERATE;   // nothing left to reuse
    } else {
      d.assign(original + start, original + start + k);
      if ((rc = ee_verify(target, seq, d.data(), k, nullptr, &a, &nxt, nullptr))) return rc;
      st->cursor = start + a + 1;
      st->phase = a < k ? EE_PHASE_GENERATE : EE_PHASE_REUSE;
    }
  }
  if (phase == EE_PHASE_GENERATE) {
    if (!draft) {
      d.clear();
      if ((rc = ee_verify(target, seq, nullptr, 0, nullptr, &a, &nxt, nullptr))) return rc;
    } else {
      int32_t lag;
      if ((rc = align_draft(target, seq, draft, dseq, out, n_out, &lag))) return rc;
      d.resize(p->gamma);
      // catch up with the output (the last `lag` tokens), giving the first draft token
      if ((rc = ee_extend(draft, dseq, out + (n_out - lag), lag, &d[0]))) return rc;
      st->draft_forwards += 1;
      for (int32_t i = 1; i < p->gamma; ++i) {
        int32_t a0;
        if ((rc = ee_verify(draft, dseq, nullptr, 0, nullptr, &a0, &d[i], nullptr))) return rc;
        st->draft_forwards += 1;
      }
      st->draft_tokens += p->gamma;
      if (p->top_k == 0) {
        rc = ee_verify(target, seq, d.data(), p->gamma, nullptr, &a, &nxt, nullptr);
      } else {
        rc = ee_verify_topk(target, 1, &seq, d.data(), p->gamma, p->top_k, p->dynamic, &a, &nxt, nullptr);
      }
      if (rc) return rc;
      // the draft holds prompt + out[0..m] + d_1..d_{gamma-1}; keep the accepted part
      if (a < p->gamma && (rc = ee_kv_rollback(draft, dseq, tl + 1 + a, nxt))) return rc;
    }
    st->phase = EE_PHASE_GENERATE;
  }
  // emit
  for (int32_t i = 0; i < a; ++i) out[n_out + i] = d[i];
  out[n_out + a] = nxt;
  *n_new = a + 1;
  st->last_phase = phase;
  st->last_accept = a;
  st->steps[phase] += 1;
  st->emitted[phase] += a + 1;
  if (phase == EE_PHASE_GENERATE) {
    int32_t ds;
    if ((rc = match(out, n_out + a + 1, original, n_orig, st->cursor, p, &ds))) return rc;
    if (ds >= 0) st->phase = EE_PHASE_REUSE;
  }
  return EE_OK;
}

}  // extern "C"
