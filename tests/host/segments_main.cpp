// Prints choose_segments(waves_base, L, resident, simds) for each input line
// "waves_base L resident simds" as "nseg seg_len pieces"; host code only, no GPU call.
#include <cstdio>

#include "scan_tiled.hpp"

int main() {
    long long wb, L, res, simds;
    while (std::scanf("%lld %lld %lld %lld", &wb, &L, &res, &simds) == 4) {
        int64_t seg_len = L, pieces = 1;
        const int64_t nseg = mbs::tiled::choose_segments(wb, L, res, simds, &seg_len, &pieces);
        std::printf("%lld %lld %lld\n", (long long)nseg, (long long)seg_len, (long long)pieces);
    }
    return 0;
}
