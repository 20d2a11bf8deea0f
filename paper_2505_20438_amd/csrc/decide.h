// The per-sequence token decision and on-device stop test (Sec. 3.3, Sec. 3.4,
// Sec. 4.4).  Runs in the single workgroup that finalises the LM-head argmax.
#pragma once
#include "device_common.h"
#include "ham_internal.h"

namespace ham {

enum { STOP_HEAD = 0, STOP_TOKEN = 1, STOP_FORCED = 2, STOP_FORCED_TOKEN = 3 };

// Decision k of sequence b: greedy token t (lowest id among equal maxima) and
// stop logit s.  Appends the token (the teacher's under teacher forcing) to the
// group, then ends the group if the stop test fires, the group is full, or the
// budget is spent.  In TOKEN mode a reserved id at k >= 1 ends the group and is
// not emitted; FORCED_TOKEN takes decision k = forced length (k >= 1) as that
// id.  Finished groups update the counters used by ham_kv_stats.
__device__ inline void decide_one(const DecideArgs& d, int b, int t, float s) {
  const SeqPtrs& st = d.st;
  if (!st.active[b]) return;
  const int k = d.k;
  d.out_tokens[b * 4 + k] = t;
  if (d.dbg_stop) d.dbg_stop[b] = s;
  bool finish;
  if ((d.mode == STOP_TOKEN && k >= 1 && t == d.stop_id) ||
      (d.mode == STOP_FORCED_TOKEN && k >= 1 && k >= st.forced[b])) {
    finish = true;
  } else {
    int tin = d.has_teacher ? st.teacher[b * 4 + k] : t;
    if (tin < 0 || tin >= d.V) {  // invalid teacher token: flag it and keep the model's own
      st.err[b] |= 4;
      tin = t;
    }
    int n = st.grp_n[b];
    st.grp_tok[b * 4 + n] = tin;
    n += 1;
    st.grp_n[b] = n;
    const int e = st.emitted[b] + 1;
    st.emitted[b] = e;
    const int bud = st.budget[b];
    finish = (d.mode == STOP_HEAD && s > d.tau) || (d.mode == STOP_FORCED && k + 1 >= st.forced[b]) ||
             n >= d.G || (bud > 0 && e >= bud);
  }
  if (finish) {
    const int n = st.grp_n[b];
    d.out_lens[b] = n;
    st.groups[b] += 1;
    st.hist[b * 5 + n] += 1;
    const int bud = st.budget[b];
    st.done[b] = (bud > 0 && st.emitted[b] >= bud) ? 1 : 0;
    st.active[b] = 0;
  }
}

}  // namespace ham
