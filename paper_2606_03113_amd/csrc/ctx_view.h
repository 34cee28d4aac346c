// What the policy trainer (dqn.cpp) reads from and writes into a decoding
// context (runtime.cpp).  Not part of the public C ABI.
#pragma once
#include "../../include/lede.h"

namespace lede {

// The device decision log of the context's last exit-policy step
// (POLICY_LOG floats per decision) with its exit layer and acceptance.
// LEDE_E_STATE unless the last step of the context was an exit-policy step
// not taken yet; a successful call takes it (a second call fails).
struct PolicyStepView {
  const float* log;
  int n_dec, l_star, accepted, n_layers;
};
int policy_step_take(lede_ctx* c, PolicyStepView* v);

// The exit-policy Q-network's device weights (W1 [H][3], b1 [H], W2 [2][H],
// b2 [2] fp32).  LEDE_E_STATE when the context has no exit policy.
struct ExitWeightsView {
  float *w1, *b1, *w2, *b2;
  int hidden;
};
int exit_weights_view(lede_ctx* c, ExitWeightsView* v);

}  // namespace lede
