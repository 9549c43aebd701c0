// HogBatch with the K negatives shared by a group of G consecutive targets
// of a sentence (the sharing of Sec. 1.1 widened from one target's input
// words to several targets). The members of a group (its targets that form
// a minibatch) take the negatives drawn at the group's first retained
// position; every member's step reads the rows as they were before the
// group, so the whole group is one snapshot step over the union of the
// members' input rows and of their targets and the shared negatives. Rows
// are staged deduplicated; per distinct input row the group keeps its
// multiplicity in every member's window, per distinct output column which
// members have it as their target and how many negative draws equal it.
#pragma once

#include "device_common.h"
#include "sgns_core.h"

namespace w2v {

constexpr int kMaxGroup = 8;  // the host also bounds 2 window G <= 64

struct GroupLds {
  int occ_id[kWave];                   // input occurrences: word
  int occ_g[kWave];                    // ... and member index
  float m[kMaxInputs][kMaxGroup];      // multiplicity of input row i in member g
  float alpha[kMaxGroup];              // learning rate of member g (0: none)
  int cand_id[kWave];                  // output candidates: word
  uint32_t tbits[kMaxOutputs];         // bit g: the column is member g's target
  float negw[kMaxOutputs];             // shared negative draws equal to it
};

// Error of slot (li, lk): sum over members g of m[li][g] alpha_g times
// sigma(-x) where the column is g's target (label 1), else -negw sigma(x)
// (label 0; a negative equal to g's own target is masked for g).
struct GroupError {
  const GroupLds* gl;
  int G;
  __device__ __forceinline__ float operator()(const MinibatchLds&, int li,
                                              int lk, float x, float,
                                              bool want_loss,
                                              float& loss_part) const {
    const float sp = 1.f / (1.f + __expf(x));    // sigma(-x)
    const float sn = 1.f / (1.f + __expf(-x));   // sigma(x)
    const uint32_t tb = gl->tbits[lk];
    const float nw = gl->negw[lk];
    float e = 0.f, l_t = 0.f, l_n = 0.f;
    for (int g = 0; g < G; ++g) {
      const float mg = gl->m[li][g];
      if (mg == 0.f) continue;
      if ((tb >> g) & 1u) {
        e += mg * gl->alpha[g] * sp;
        l_t += mg;
      } else {
        e -= mg * gl->alpha[g] * nw * sn;
        l_n += mg * nw;
      }
    }
    if (want_loss) {
      if (l_t != 0.f) loss_part += l_t * softplus(-x);
      if (l_n != 0.f) loss_part += l_n * softplus(x);
    }
    return e;
  }
};

}  // namespace w2v
