// Sort keys of the dispatch policies and of the calibration partition.
#pragma once

#include "common.h"
#include "kernels.h"

namespace ds {

// The (key, value) pair of position j of the sequence a sort reorders:
//   Fifo    key = ordered(arrival[j]),             value j
//   Budget  key = ordered(budget[fifo[j]]),        value fifo[j]
//   Aging   key = ordered(aged score of fifo[j]),  value fifo[j]
//   Class   key = priority class of tier,          value fifo[j]
//   Tier    key = tier,                            value fifo[j]
//   Group   key = group[j],                        value j
// The aged score is max(floor, p - rate * max(0, t_now - arrival)) with each
// operation rounded separately (no fused multiply-add). key_out, if given,
// receives each request's primary key.
__device__ __forceinline__ void produce(const SortInput &in, SortKind kind, double *key_out,
                                        uint32_t n, uint32_t j, uint64_t &k, uint32_t &v)
{
    switch (kind) {
    case SortKind::Fifo: {
        double a = in.arrival[j];
        k = ordered_bits(a);
        v = j;
        if (key_out) key_out[j] = a;
        break;
    }
    case SortKind::Budget: {
        uint32_t i = in.fifo[j];
        i = i < n ? i : 0;
        double b = in.budget[i];
        k = ordered_bits(b);
        v = i;
        if (key_out) key_out[i] = b;
        break;
    }
    case SortKind::Aging: {
        uint32_t i = in.fifo[j];
        i = i < n ? i : 0;
        uint32_t q = in.tier[i];
        q = q < 16 ? q : 15;
        double w = in.t_now - in.arrival[i];
        if (w < 0.0) w = 0.0;
        double d = in.aging_rate * w;
        double e = in.prio[q] - d;
        if (e < in.aging_floor) e = in.aging_floor;
        k = ordered_bits(e);
        v = i;
        if (key_out) key_out[i] = e;
        break;
    }
    case SortKind::Class: {
        uint32_t i = in.fifo[j];
        i = i < n ? i : 0;
        uint32_t q = in.tier[i];
        q = q < 16 ? q : 15;
        k = in.cls[q];
        v = i;
        if (key_out) key_out[i] = in.prio[q];
        break;
    }
    case SortKind::Tier: {
        uint32_t i = in.fifo[j];
        i = i < n ? i : 0;
        uint32_t q = in.tier[i];
        k = q < 16 ? q : 15;
        v = i;
        break;
    }
    default: {   // Group
        k = in.group[j];
        v = j;
        break;
    }
    }
}

}  // namespace ds
