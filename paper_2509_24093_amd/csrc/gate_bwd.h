// Internal interface of the backward of the gating and value tensor product
// (gate.hip), beside the forward's GateArgs.
#pragma once

#include <hip/hip_runtime.h>

namespace cgconv {

// Given G = dL/df for f = gate_value(u, v), all fp32 [B][N][K][C]:
//   a = g u, da = R-transposed contraction of (G, v), dv = that of (G, a),
//   h[b,i,l,c] = g sum_m u da (the gate's gradient times g),
//   S[b,l,c] = sum_i h[b,i,l,c],  du = g da + (h - g S) u / ||u_l||.
struct GateBwdArgs {
  const float* u;
  const float* v;
  const float* G;
  float* du;             // or nullptr (then h, S are not formed)
  float* dv;             // or nullptr
  float* h;              // [B][N][L+1][C]
  float* psum;           // [B][chunks][L+1][C]: sums of h over token chunks
  float* S;              // [B][L+1][C]
  float2* part;          // softmax partials and statistics, as in the forward
  float2* fin;
  const float* scales;   // [6][K]: the backward scales (first operand: 0..3K, second: 3K..6K)
  int B, N, C;
  hipEvent_t* events;    // optional: 5 events around the four stages
};
template <int L>
hipError_t launch_gate_backward(const GateBwdArgs& a, hipStream_t s);

}  // namespace cgconv
