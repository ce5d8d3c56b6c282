// plan.hpp -- host-only planning of a step: validation, tile tables,
// workspace layout and coefficients.  No HIP calls.
#pragma once
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/rikfad.h"
#include "layout.hpp"

namespace rk {

struct Plan {
    std::vector<TensorDesc> tensors;
    std::vector<const void *> grads;
    std::vector<Tile> tiles;          // grouped by storage type; see TileGroup
    std::vector<TileGroup> groups;    // one launch each (per storage type and width)
    int64_t matrix_tiles = 0;
    std::vector<FinItem> fin;         // row items, then column items
    int64_t row_items = 0;
    int32_t fin_log2 = kFinSmallLog2; // log2 of the finalisation workgroup size
    int64_t ws_floats = 0;            // partial-sum workspace (floats)
    int64_t matrices = 0, vectors = 0, elements = 0;
    int64_t state_bytes = 0, ikfad_state_bytes = 0, min_bytes = 0, stream_min_bytes = 0;
};

// Validates and plans an R-iKFAD context.  Returns RIKFAD_OK or an error
// code with a message in `err`.
// rows_per_wave > 0 fixes the rows per wave of every matrix tile (narrow
// blocks still scale it up); 0 takes kRowsPerWave, halved for sets with
// fewer matrix tiles than the chip has compute units.
rikfad_status plan_rikfad(const rikfad_tensor *t, int64_t count, Plan &out, std::string &err,
                          int rows_per_wave = 0);

// Validates and plans a full-tensor iKFAD context (every tensor element-wise).
rikfad_status plan_ikfad(const ikfad_tensor *t, int64_t count, Plan &out, std::string &err);

rikfad_status check_hparams(const rikfad_hparams *hp, std::string &err);
Coeffs make_coeffs(const rikfad_hparams &hp);

// Access width (elements per lane) usable for a gradient pointer of a tensor
// planned with width `vec`; false if the pointer breaks that alignment.
bool grad_fits(const void *g, int32_t dtype, int32_t vec);

}  // namespace rk
