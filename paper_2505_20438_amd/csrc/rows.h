// Row -> (sequence, KV slot, RoPE position, visible slots) for every kind of
// launch of the decode loop.
#pragma once
#include "ham_internal.h"

namespace ham {

struct RowInfo {
  int b, slot, pos, n_valid, enabled;
};

__device__ __forceinline__ RowInfo row_info(const RowMap& rm, int r) {
  RowInfo ri;
  switch (rm.mode) {
    case ROWS_PREFILL:  // one slot per input row, causal; position = slot unless given
      ri.b = rm.b;
      ri.slot = rm.t0 + r;
      ri.pos = rm.pos ? rm.pos[(size_t)rm.b * rm.ldpos + ri.slot] : ri.slot;
      ri.n_valid = ri.slot + 1;
      ri.enabled = 1;
      break;
    case ROWS_DECODE:  // one fused input per running sequence, at its group's last position
      ri.b = r;
      ri.slot = rm.st.cur_slot[r];
      ri.pos = rm.st.cur_pos[r];
      ri.n_valid = rm.st.kv_len[r];
      ri.enabled = rm.st.step_on[r];
      break;
    case ROWS_MICRO1: {  // context rows then the first token, local positions 0..C
      const int c = r % (rm.C + 1);
      ri.b = r / (rm.C + 1);
      ri.slot = c;
      ri.pos = c;
      ri.n_valid = c + 1;
      ri.enabled = rm.st.active[ri.b];
      break;
    }
    default: {  // ROWS_MICROK: the token of micro step k-1 at local position C+k-1
      ri.b = r;
      ri.slot = rm.C + rm.k - 1;
      ri.pos = ri.slot;
      ri.n_valid = ri.slot + 1;
      ri.enabled = rm.st.active[r];
      break;
    }
  }
  return ri;
}

}  // namespace ham
