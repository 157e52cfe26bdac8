// Compute accounting of a precision schedule, next to its measured time:
// the paper's Eff. W-bit and Rel. BitOPs (Sec. 4, quality-compute table) and
// the bit-serial engine's cycle laws (Sec. 3.3 / 4.3: cycles grow with the
// product of weight and activation planes, switching precision costs
// nothing; per-tile totals at four activation planes for the
// activation-stationary dataflow grow as 570 L + 2603).  Host arithmetic
// over the same layer list and table as tasq_run_schedule.
#include "tasq.h"

#include <cstring>

namespace {

// Activation-stationary tile law at R = 4 activation planes (Tab. codesign).
constexpr double kAsSlope = 570.0;
constexpr double kAsIntercept = 2603.0;

int stage_of(int t, int S, int T) { return (int)(((long long)t * S) / T); }

}  // namespace

extern "C" int tasq_schedule_cost(const tasq_layer *layers, int L, const uint8_t *b_table, int S,
                                  int T, int t_begin, int t_end, int act_bits, tasq_cost *out)
{
    if (!out)
        return TASQ_ERR_NULL;
    std::memset(out, 0, sizeof *out);
    if (L < 0 || S < 1 || T < 1 || S > T || t_begin < 0 || t_end > T || t_begin > t_end ||
        act_bits < 1 || act_bits > 16)
        return TASQ_ERR_RANGE;
    if (L > 0 && (!layers || !b_table))
        return TASQ_ERR_NULL;
    for (int l = 0; l < L; ++l) {
        const tasq_layer &ly = layers[l];
        if (ly.M < 0 || ly.N < 0 || ly.K < 0)
            return TASQ_ERR_DIM;
        for (int s = 0; s < S; ++s)
            if (b_table[l * S + s] < 1 || b_table[l * S + s] > 8)
                return TASQ_ERR_BITS;
    }
    // Sums in double: MAC counts of a whole schedule stay far below 2^53.
    double macs = 0, bw = 0, cas = 0, bsum = 0, count = 0;
    for (int t = t_begin; t < t_end; ++t) {
        const int s = stage_of(t, S, T);
        for (int l = 0; l < L; ++l) {
            const double mac = (double)layers[l].M * (double)layers[l].N * (double)layers[l].K;
            const int b = b_table[l * S + s];
            macs += mac;
            bw += mac * b;
            cas += mac * (kAsSlope * b + kAsIntercept);
            bsum += b;
            count += 1;
        }
    }
    out->macs = macs;
    out->b_mean = count > 0 ? bsum / count : 0.0;
    out->bitops = bw * act_bits;
    if (macs > 0) {
        out->b_eff = bw / macs;
        out->rel_bitops = bw * act_bits / (64.0 * macs);
        out->rel_cycles_measured = bw / (8.0 * macs);
        out->rel_cycles_as_a4 = cas / (macs * (kAsSlope * 8 + kAsIntercept));
    }
    return TASQ_OK;
}
