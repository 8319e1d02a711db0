// The stored half of the triple table of the ternary 3-in-5 format (LUT Tensor
// Core, Section 5 with the symmetry of Eq. 4): entry i < 14 is the dot product of
// activations x0..x2 with the pattern v = 13 + i, w_e = (base-3 digit e of v) - 1
// with the first activation most significant, i.e. the patterns
//   i:  0        1        2         3        4        5          6         7
//       (0,0,0)  (0,0,1)  (0,1,-1)  (0,1,0)  (0,1,1)  (1,-1,-1)  (1,-1,0)  (1,-1,1)
//   i:  8         9        10       11        12       13
//       (1,0,-1)  (1,0,0)  (1,0,1)  (1,1,-1)  (1,1,0)  (1,1,1)
// and pattern 13 - i is its negation.  Every entry is formed as
// (w0 x0 + w1 x1) + w2 x2 with zero terms dropped, 10 additions in all; the
// precompute kernel and the fused kernel share this function, so their FP
// tables are bitwise equal.
#pragma once

#include <hip/hip_runtime.h>

namespace lutgemm {

template <typename T>
__device__ __forceinline__ void tri_table14(T x0, T x1, T x2, T (&e)[14]) {
    const T p = x0 + x1, m = x0 - x1;
    e[0] = T(0);
    e[1] = x2;
    e[2] = x1 - x2;
    e[3] = x1;
    e[4] = x1 + x2;
    e[5] = m - x2;
    e[6] = m;
    e[7] = m + x2;
    e[8] = x0 - x2;
    e[9] = x0;
    e[10] = x0 + x2;
    e[11] = p - x2;
    e[12] = p;
    e[13] = p + x2;
}

}  // namespace lutgemm
