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
#include "kernel_args.h"
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

// One group step. Every output row stays in registers (o, and its update
// go) while the distinct input rows go by in blocks of IB = 64 / OMAX: per
// block, the IB x OMAX logits come from one transposing reduction, the
// block's input rows take their complete update at once, and the output
// updates accumulate until every block is done. All rows are read before
// any of them is written (input rows are distinct, and M_in and M_out are
// different matrices), so this is the snapshot step of the group.
template <int C, int OMAX>
__device__ __forceinline__ void run_group(const EpochArgs& a, int lane,
                                          int n_in, int n_out,
                                          MinibatchLds& mb, const GroupLds& gl,
                                          int G, bool want_loss,
                                          float& loss_part) {
  constexpr int IB = kWave / OMAX;
  constexpr int kSlots = IB * OMAX;
  const RowTiers<C, false> io{a.part, a.split_rows, a.hot_rows, a.ld, a.D, lane};
  const GroupError err{&gl, G};
  float o[OMAX][C], go[OMAX][C];
#pragma unroll
  for (int k = 0; k < OMAX; ++k) {
#pragma unroll
    for (int c = 0; c < C; ++c) go[k][c] = 0.f;
    if (k < n_out) {
      const int id = uniform_int(mb.out[k]);
      load_row<C, true>(a.M_out, id, a.ld, a.D, lane, o[k]);
      io.add_split(1, id, o[k]);
    } else {
#pragma unroll
      for (int c = 0; c < C; ++c) o[k][c] = 0.f;
    }
  }
  for (int i0 = 0; i0 < n_in; i0 += IB) {
    float av[IB][C];
#pragma unroll
    for (int ii = 0; ii < IB; ++ii) {
      if (i0 + ii < n_in) {
        const int id = uniform_int(mb.ctx[i0 + ii]);
        load_row<C, true>(a.M_in, id, a.ld, a.D, lane, av[ii]);
        io.add_split(0, id, av[ii]);
      } else {
#pragma unroll
        for (int c = 0; c < C; ++c) av[ii][c] = 0.f;
      }
    }
    auto partial = [&](int s) -> float {
      const int ii = s / OMAX;
      const int k = s % OMAX;
      if (s >= kSlots || i0 + ii >= n_in || k >= n_out) return 0.f;
      float acc = 0.f;
#pragma unroll
      for (int c = 0; c < C; ++c) acc = fmaf(av[ii][c], o[k][c], acc);
      return acc;
    };
    const float x = xpose_reduce64_lazy(partial, lane);
    const int li = i0 + lane / OMAX;
    const int lk = lane % OMAX;
    const bool valid = lane < kSlots && li < n_in && lk < n_out;
    float e_lane = 0.f;
    if (valid) e_lane = err(mb, li, lk, x, 0.f, want_loss, loss_part);

#pragma unroll
    for (int ii = 0; ii < IB; ++ii) {
      if (i0 + ii < n_in) {
        float g[C];
#pragma unroll
        for (int c = 0; c < C; ++c) g[c] = 0.f;
#pragma unroll
        for (int k = 0; k < OMAX; ++k) {
          if (k < n_out) {
            const float e = lane_value(e_lane, ii * OMAX + k);
#pragma unroll
            for (int c = 0; c < C; ++c) {
              g[c] = fmaf(e, o[k][c], g[c]);
              go[k][c] = fmaf(e, av[ii][c], go[k][c]);
            }
          }
        }
        io.update(0, a.M_in, uniform_int(mb.ctx[i0 + ii]), av[ii], g);
      }
    }
  }
#pragma unroll
  for (int k = 0; k < OMAX; ++k)
    if (k < n_out) io.update(1, a.M_out, uniform_int(mb.out[k]), o[k], go[k]);
}

}  // namespace w2v
