// The MLP's last layer with Heun's Euler prediction as its epilogue.
#pragma once

#include "pd_internal.h"

namespace pd {

// Heun's first stage (the Euler step of the DDIM ODE, Sec. 3.3) on the rows of
// the current window: xt[j] = x_{t+j} + (A_{t+j} x_{t+j} + B_{t+j} eps[j]),
// with x_{t+j} read from the ring as the scan reads it (slot (m <= f ? m : f)
// mod ring_slots for m = t + j).  Rows are window rows of `group` samples each
// (j = row / group), as the loop's row source lays them out.
struct HeunPredictArgs {
    const LoopState* st;   // the iteration's loop state (t, f)
    const float* ring;     // [ring_slots][B * D]
    const float* A;        // [T] drift coefficients
    const float* B;
    int32_t ring_slots;
    float* xt;             // [p][B * D] predictions
};

// The last layer of the MLP (dense input x, [rows][K]) into y, and each
// output's Euler prediction into h.xt.  y and h.xt hold what
// launch_linear_dense and the separate prediction kernel give, bit for bit.
void launch_linear_dense_predict(const LinearArgs& a, const float* x, const RowSrc& rows,
                                 const HeunPredictArgs& h, float* y, hipStream_t s);

}  // namespace pd
