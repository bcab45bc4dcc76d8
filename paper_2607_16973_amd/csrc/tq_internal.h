// Internal declarations shared by the host-side translation units of libtq.
#pragma once

#include <cstdint>
#include <mutex>
#include <string>
#include <vector>

#include "tq.h"

namespace tq {

// ------------------------------------------------------------------ errors
void set_error(const std::string &msg);
tq_status fail(tq_status st, const std::string &msg);

// ----------------------------------------------------------------- codebook
// Lloyd-Max tables for the sphere-coordinate law in R^d (host, float64).
struct CodebookTables {
    int d = 0;
    int bits = 0;
    std::vector<double> bounds;  // L-1, increasing, bounds[L/2-1] == 0
    std::vector<double> cents;   // L, increasing, antisymmetric
    double mse = 0.0;            // per-coordinate distortion
};
// Returns false (with set_error) if the solver fails.
bool solve_lloyd_max(int d, int bits, CodebookTables *out);

// ----------------------------------------------------------------- rotation
// Haar orthogonal matrix for (d, seed), float32 row-major (host).
bool make_rotation(int d, uint64_t seed, std::vector<float> *R32);

// -------------------------------------------------------------------- index
// Whether the index's rotation is already on the current device.
bool index_rotation_resident(const tq_index *x);

}  // namespace tq

// Opaque handle definitions (C ABI types).
struct tq_codebook {
    tq::CodebookTables t;
};

struct tq_rotation {
    int d = 0;
    uint64_t seed = 0;
    std::vector<float> R;         // d*d row-major
    mutable std::mutex mu;        // guards the lazily created device copy
    mutable float *R_dev = nullptr;
    mutable int R_dev_device = -1;
};
