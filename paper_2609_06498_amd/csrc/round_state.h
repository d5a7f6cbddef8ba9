// Per-sequence round state shared by the acceptance kernels (greedy and
// speculative sampling): the carry record and the outcome writer.
#pragma once
#include <hip/hip_runtime.h>

namespace dflow {

// carry record per sequence: [last relayed block index, a + 1, bonus, first
// rejected proposal, first relayed block index]; block index i (first <= i <=
// last) takes verify row rec[1] + i - 1 = a + i
constexpr int CARRY_REC = 5;

// Outcome of a round for sequence s with a accepted drafts and token b at block
// index a+1 (bonus or correction): committed = d_1..d_a, b (rest -1); the
// carried rows go to next-round block indices lo..hi by the window:
// 0 suffix 1..K-1-a, 1 suffix+tail 1..K-a, 2 suffix-inputs 2..K-a.
__device__ inline void write_accept_outcome(int s, int a, int b, const int* blk, int B, int carry_window,
                                            int* accept_len, int* bonus, int* committed, int* n_carry,
                                            int* carry_rec) {
  const int K = B - 1;
  for (int j = 0; j < B; ++j) committed[(size_t)s * B + j] = j < a ? blk[j + 1] : (j == a ? b : -1);
  const int lo = carry_window == 2 ? 2 : 1;
  const int hi = carry_window == 0 ? K - 1 - a : K - a;
  const int n = hi >= lo ? hi - lo + 1 : 0;
  accept_len[s] = a;
  if (bonus) bonus[s] = b;
  if (n_carry) n_carry[s] = n;
  int* rec = carry_rec + (size_t)s * CARRY_REC;
  rec[0] = n > 0 ? hi : 0;
  rec[1] = a + 1;
  rec[2] = b;
  rec[3] = a < K ? blk[a + 1] : -1;
  rec[4] = lo;
}

}  // namespace dflow
