// Host-side figures for `bench.py --suite`: what one geot_select call costs
// (median over 20 batches of 50,000 calls, 10^6 in all, over four shapes; with
// and without index statistics), and the HBM peak the device properties imply
// (memory clock x bus width, at 2 and at 4 transfers per clock).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cstdio>
#include <vector>

#include "geot.h"

int main() {
    const int64_t shapes[4][4] = {{114615892, 232965, 32, 0}, {61859140, 2449029, 128, 1},
                                  {65536, 4096, 32, 0}, {2000000, 100000, 8, 0}};
    geot_index_stats_t st = {114615892, 232965, 87791, 0, 0, 492.0, 884.0 * 884.0};
    geot_kernel_choice_t c;
    for (int with_stats = 0; with_stats < 2; ++with_stats) {
        std::vector<double> ns;
        for (int rep = 0; rep < 20; ++rep) {
            const auto t0 = std::chrono::steady_clock::now();
            for (int i = 0; i < 50000; ++i) {
                const int64_t *s = shapes[i & 3];
                if (geot_select(s[0], s[1], s[2], GEOT_OP_SUM, (int32_t)s[3], with_stats ? &st : nullptr, &c) !=
                    GEOT_SUCCESS)
                    return 1;
            }
            const auto t1 = std::chrono::steady_clock::now();
            ns.push_back(std::chrono::duration<double, std::nano>(t1 - t0).count() / 50000.0);
        }
        std::sort(ns.begin(), ns.end());
        std::printf("{\"suite\": \"geot_select host time per call%s\", \"ns\": %.1f, \"calls\": 1000000}\n",
                    with_stats ? " (with index statistics)" : "", ns[ns.size() / 2]);
    }
    int clk = 0, bus = 0;
    if (hipDeviceGetAttribute(&clk, hipDeviceAttributeMemoryClockRate, 0) != hipSuccess ||
        hipDeviceGetAttribute(&bus, hipDeviceAttributeMemoryBusWidth, 0) != hipSuccess)
        return 2;
    // HBM3E moves more than two bits per pin per reported memory clock: both readings are printed
    std::printf("{\"suite\": \"HBM peak from device properties\", \"memory_clock_khz\": %d, \"bus_width_bits\": %d, "
                "\"GB/s at 2 transfers per clock\": %.1f, \"GB/s at 4 transfers per clock\": %.1f}\n",
                clk, bus, 2.0 * clk * 1e3 * bus / 8.0 / 1e9, 4.0 * clk * 1e3 * bus / 8.0 / 1e9);
    return 0;
}
