// The LSTM cell of the recurrent models (section 4.1): no bias, gate order
// (i, f, g, o),
//     c' = sigmoid(f) * c + sigmoid(i) * tanh(g),   h' = sigmoid(o) * tanh(c').
// Shared by the cell kernel of the two-kernel step and the fused step kernel, so
// both apply the same arithmetic to the gate pre-activations.
#pragma once

#include <hip/hip_runtime.h>

namespace darb {

__device__ __forceinline__ float lstm_sigmoid(float z) { return 1.0f / (1.0f + __expf(-z)); }

// gi, gf, gg, go: gate pre-activations; c: the cell state, updated; returns h'.
__device__ __forceinline__ float lstm_cell(float gi, float gf, float gg, float go, float &c) {
    const float cn = lstm_sigmoid(gf) * c + lstm_sigmoid(gi) * tanhf(gg);
    c = cn;
    return lstm_sigmoid(go) * tanhf(cn);
}

}  // namespace darb
