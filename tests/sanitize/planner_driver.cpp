// Host-only driver of the circuit intake and the tile-pass planner, built
// with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_sanitizers.py. It reads circuits from a binary file and runs
// build_circuit (which plans both dtypes) under several planner options.
//
// File: repeated records of int32 n, n_gates, n_inputs, n_weights, embed,
// embed_first, n_channels, expect_ok, then n_gates * 5 int32 gate fields and
// n_channels * 3 float64 channel probabilities.
#include <cstdio>
#include <cstring>
#include <vector>

#include "plan.hpp"

using namespace qlayer;

int main(int argc, char** argv) {
    if (argc < 2) return 2;
    FILE* f = std::fopen(argv[1], "rb");
    if (!f) return 2;
    int n_cases = 0, n_plans = 0, n_rejected = 0;
    for (;;) {
        int32_t hdr[8];
        if (std::fread(hdr, sizeof(int32_t), 8, f) != 8) break;
        const int n = hdr[0], G = hdr[1], F = hdr[2], P = hdr[3], nch = hdr[6], expect_ok = hdr[7];
        std::vector<int32_t> g((size_t)G * 5);
        std::vector<double> pp((size_t)nch * 3);
        if (G && std::fread(g.data(), sizeof(int32_t), g.size(), f) != g.size()) return 3;
        if (nch && std::fread(pp.data(), sizeof(double), pp.size(), f) != pp.size()) return 3;
        Extras ext;
        ext.embed = hdr[4];
        ext.embed_first = hdr[5];
        ext.pauli_p = nch ? pp.data() : nullptr;
        // the beam search (the default) on the plain options; the plans of many
        // passes take the look-ahead alone, which keeps the sanitized run short
        const Options variants[] = {
            Options{},
            [] { Options o; o.pass_search = -1; o.product_prefix = -1; o.cz_groups = -1; return o; }(),
            [] { Options o; o.rz_groups = -1; o.max_gates_per_pass = 7; o.pass_search = 1; o.product_prefix = 1; return o; }(),
            [] { Options o; o.log_regs = 3; o.log_threads = 7; o.low_qubits = 2; o.pass_search = 1; return o; }(),
            [] { Options o; o.force_tiled = -1; return o; }(),
        };
        for (const Options& o : variants) {
            Circuit c;
            const std::string err = build_circuit(n, g.data(), G, F, P, ext, o, c);
            if (err.empty()) {
                n_plans++;
                if (!expect_ok) {
                    std::printf("case %d: accepted an invalid circuit\n", n_cases);
                    return 4;
                }
            } else {
                n_rejected++;
                if (expect_ok && err.compare(0, 7, "option:") != 0 && err != "circuit too small for the tile kernel") {
                    std::printf("case %d: rejected: %s\n", n_cases, err.c_str());
                    return 5;
                }
            }
        }
        n_cases++;
    }
    std::printf("cases %d plans %d rejected %d\n", n_cases, n_plans, n_rejected);
    return 0;
}
