// Parallel decoding scheduler: host-only C++ (no device code).
//
// Decides, round by round, what the target verifies and what the draft drafts
// in the pipeline of pre-verify and post-verify rounds, and keeps the committed
// output, the pending (drafted, unverified) window and the draft's rollback
// point.  The caller runs the two models, typically on two HIP streams, and
// reports the target's verdict; the scheduler launches nothing.
//
// State machine.  The pending window is what the next round verifies:
//   startup    the draft's first token d0 is decided against the target's
//              prefill output (no forward, no time); d1..d_gamma, drafted during
//              prefill, stay pending.
//   pre        pending is empty: the draft drafts gamma tokens from the
//              committed prefix and the target verifies the first of them.
//   post       the target verifies the whole pending window while the draft
//              drafts gamma tokens after it.
// All verified tokens accepted: they are committed, the rest become pending
// and the next round is post (pre if nothing is pending).  A rejection
// commits the accepted prefix and the target's token, drops every other
// draft, sets the rollback point just before the target's token and makes the
// next round pre.  A round that runs forwards lasts max(gamma, c) t.
#include <algorithm>
#include <new>
#include <vector>

#include "pvlm.h"

struct pvlm_pd {
  int gamma = 0;
  double c = 0.0;
  int max_len = 0;
  bool started = false;
  bool startup_round = true;      // the free pre-verify of d0 is next
  std::vector<int32_t> out;       // committed tokens
  std::vector<int32_t> pending;   // drafted, not yet verified
  int32_t run = 0, max_run = 0;   // committed draft tokens since the last target token
  int32_t rounds = 0;             // rounds that ran forwards
  int32_t keep = 0;               // last rollback point
  double clock = 0.0;
};

namespace {

constexpr int kMaxGamma = 1024;
constexpr int kMaxLen = 1 << 26;

bool done(const pvlm_pd* pd) { return static_cast<int>(pd->out.size()) >= pd->max_len; }

void make_plan(const pvlm_pd* pd, pvlm_pd_round* r) {
  const int32_t n = static_cast<int32_t>(pd->out.size());
  const int32_t np = static_cast<int32_t>(pd->pending.size());
  r->verify_begin = n;
  if (done(pd)) {
    r->mode = PVLM_PD_DONE;
    r->verify_count = r->draft_count = 0;
    r->draft_begin = n;
    r->cost = 0.0;
  } else if (pd->startup_round) {
    r->mode = PVLM_PD_PRE_VERIFY;
    r->verify_count = 1;
    r->draft_begin = n + np;
    r->draft_count = 0;
    r->cost = 0.0;
  } else if (np == 0) {
    r->mode = PVLM_PD_PRE_VERIFY;
    r->verify_count = 1;
    r->draft_begin = n;
    r->draft_count = pd->gamma;
    r->cost = std::max(static_cast<double>(pd->gamma), pd->c);
  } else {
    r->mode = PVLM_PD_POST_VERIFY;
    r->verify_count = np;
    r->draft_begin = n + np;
    r->draft_count = pd->gamma;
    r->cost = std::max(static_cast<double>(pd->gamma), pd->c);
  }
}

pvlm_status copy_out(const std::vector<int32_t>& v, int32_t* dst, int cap, int* n) {
  if (!n) return PVLM_ERR_NULL;
  *n = static_cast<int>(v.size());
  if (cap == 0 && !dst) return PVLM_OK;  // size query
  if (cap < 0) return PVLM_ERR_SHAPE;
  if (!dst) return PVLM_ERR_NULL;
  std::copy_n(v.begin(), std::min<size_t>(v.size(), static_cast<size_t>(cap)), dst);
  return static_cast<size_t>(cap) < v.size() ? PVLM_ERR_SHAPE : PVLM_OK;
}

}  // namespace

extern "C" pvlm_status pvlm_pd_create(int gamma, double c, int max_len, pvlm_pd** out) {
  if (!out) return PVLM_ERR_NULL;
  *out = nullptr;
  if (gamma < 1 || gamma > kMaxGamma || !(c > 0.0 && c < 1e300) || max_len < 1 ||
      max_len > kMaxLen)
    return PVLM_ERR_SHAPE;
  pvlm_pd* pd = new (std::nothrow) pvlm_pd;
  if (!pd) return PVLM_ERR_UNSUPPORTED;
  pd->gamma = gamma;
  pd->c = c;
  pd->max_len = max_len;
  pd->out.reserve(static_cast<size_t>(max_len) + gamma + 2);
  pd->pending.reserve(2 * static_cast<size_t>(gamma) + 1);
  *out = pd;
  return PVLM_OK;
}

extern "C" void pvlm_pd_destroy(pvlm_pd* pd) { delete pd; }

extern "C" pvlm_status pvlm_pd_start(pvlm_pd* pd, const int32_t* startup) {
  if (!pd || !startup) return PVLM_ERR_NULL;
  if (pd->started) return PVLM_ERR_SHAPE;
  pd->pending.assign(startup, startup + pd->gamma + 1);
  pd->started = true;
  return PVLM_OK;
}

extern "C" pvlm_status pvlm_pd_plan(const pvlm_pd* pd, pvlm_pd_round* round) {
  if (!pd || !round) return PVLM_ERR_NULL;
  if (!pd->started) return PVLM_ERR_SHAPE;
  make_plan(pd, round);
  return PVLM_OK;
}

extern "C" pvlm_status pvlm_pd_finish(pvlm_pd* pd, const int32_t* drafted, int n_drafted,
                                      int n_accepted, int32_t target_token) {
  if (!pd) return PVLM_ERR_NULL;
  if (!pd->started) return PVLM_ERR_SHAPE;
  pvlm_pd_round r;
  make_plan(pd, &r);
  if (r.mode == PVLM_PD_DONE || n_drafted != r.draft_count || n_accepted < 0 ||
      n_accepted > r.verify_count)
    return PVLM_ERR_SHAPE;
  if (n_drafted > 0 && !drafted) return PVLM_ERR_NULL;
  // the round's window: pre rounds verify the first new draft
  if (r.mode == PVLM_PD_PRE_VERIFY && n_drafted > 0) pd->pending.clear();
  pd->pending.insert(pd->pending.end(), drafted, drafted + n_drafted);
  pd->out.insert(pd->out.end(), pd->pending.begin(), pd->pending.begin() + n_accepted);
  pd->run += n_accepted;
  pd->max_run = std::max(pd->max_run, pd->run);
  if (n_accepted == r.verify_count) {
    pd->pending.erase(pd->pending.begin(), pd->pending.begin() + r.verify_count);
  } else {
    pd->keep = static_cast<int32_t>(pd->out.size());
    pd->out.push_back(target_token);
    pd->run = 0;
    pd->pending.clear();
  }
  pd->startup_round = false;
  pd->clock += r.cost;
  if (r.cost > 0.0) ++pd->rounds;
  return PVLM_OK;
}

extern "C" pvlm_status pvlm_pd_output(const pvlm_pd* pd, int32_t* out, int cap, int* n) {
  if (!pd) return PVLM_ERR_NULL;
  return copy_out(pd->out, out, cap, n);
}

extern "C" pvlm_status pvlm_pd_pending(const pvlm_pd* pd, int32_t* out, int cap, int* n) {
  if (!pd) return PVLM_ERR_NULL;
  return copy_out(pd->pending, out, cap, n);
}

extern "C" pvlm_status pvlm_pd_get_stats(const pvlm_pd* pd, pvlm_pd_stats* st) {
  if (!pd || !st) return PVLM_ERR_NULL;
  pvlm_pd_round r;
  make_plan(pd, &r);
  st->mode = pd->started ? r.mode : PVLM_PD_PRE_VERIFY;
  st->committed = static_cast<int32_t>(pd->out.size());
  st->pending = static_cast<int32_t>(pd->pending.size());
  st->target_rounds = pd->rounds;
  st->max_draft_run = pd->max_run;
  st->draft_keep = pd->keep;
  st->elapsed = pd->clock;
  return PVLM_OK;
}
