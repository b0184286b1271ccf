// Prints choose_segments(waves_base, L, resident) for each input line
// "waves_base L resident" as "nseg seg_len"; host code only, no GPU call.
#include <cstdio>

#include "scan_tiled.hpp"

int main() {
    long long wb, L, res;
    while (std::scanf("%lld %lld %lld", &wb, &L, &res) == 3) {
        int64_t seg_len = L;
        const int64_t nseg = mbs::tiled::choose_segments(wb, L, res, &seg_len);
        std::printf("%lld %lld\n", (long long)nseg, (long long)seg_len);
    }
    return 0;
}
