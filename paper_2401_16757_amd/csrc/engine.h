// engine.h -- internal state of a swap-engine context (not part of the ABI).
#pragma once
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/swapnet.h"

namespace sn {

constexpr int64_t kAlign = 256;   // alignment of every tensor and slab in the arena

inline int64_t align_up(int64_t v, int64_t a = kAlign) { return (v + a - 1) / a * a; }
inline int round8(int v) { return (v + 7) / 8 * 8; }

// Shape of an activation slot: rows x cols fp16 (or fp32) elements.  Image
// slots: rows = H*W, cols = Cp; token slots: rows = max tokens, cols = C.
struct Slot {
    bool used = false;
    int h = 0, w = 0;          // spatial size (image slots)
    int c = 0, cp = 0;         // channels, padded channels (cols)
    int rows = 0;
    int elem = 2;              // bytes per element
    int first = 1 << 30;       // first layer writing it (-1: network input)
    int last = -1;             // last layer reading it (L: network output)
    int64_t bytes = 0, off = 0;
};

// One layer after validation, with its device-layout tensors (host copies
// until the image is built).
struct Layer {
    sn_layer d{};
    int block = 0;
    bool token = false;        // part of a token (decoder) network
    int out_h = 1, out_w = 1;
    int cin_p = 0, cout_p = 0; // padded channel counts of src / dst
    int K = 0;                 // device row length in halves (conv, linear)
    int64_t units = 0;         // splittable output units (0: no weights)
    int rows_per_unit = 1;     // weight rows per unit (2 for SwiGLU)
    int64_t w_unit_bytes = 0;  // device weight bytes per unit
    int64_t b_unit_bytes = 0;  // device bias bytes per unit
    int kernel = -1;           // conv tile variant (image convs)
    int ksplit = 1, kps = 0;   // conv K split (see ConvPlan)
    std::vector<uint16_t> w_dev, b_dev;  // device-layout tensors
};

// A piece = output units [u0, u1) of one layer, placed in one slab.
struct Piece {
    int layer = 0;
    int64_t u0 = 0, u1 = 0;
    int64_t w_off = -1, b_off = -1;   // slab-relative
    int64_t w_bytes = 0, b_bytes = 0;
};

struct Slab {
    std::vector<int> pieces;          // indices into Ctx::pieces (after lowering)
    int64_t bytes = 0;
    int64_t image_off = 0, arena_off = 0;
    int wait = -1;                    // newest earlier slab whose arena range this
                                      // slab's swap-in overwrites (-1: none)
    int wrap = -1;                    // wait == -1: last slab of the inference that
                                      // overlaps this range; the next inference's
                                      // swap-in of this slab waits for it (-1: none)
};

// Output units [u0, u1) of one layer, before the slab layout is fixed.
struct PieceSpec {
    int layer;
    int64_t u0, u1;
};
using SlabSpec = std::vector<PieceSpec>;

struct PlanResult {
    std::vector<Piece> pieces;
    std::vector<Slab> slabs;
    bool resident = false;
    int64_t image_bytes = 0, high_water = 0;
};

// Delay model of a slab (the input / execution / output delays of Sec. 5,
// for this engine; see sn_cost_model in swapnet.h).  Times in seconds.
struct CostModel {
    double alpha = 1.0 / 56e9;   // swap-in per byte
    double beta = 14e-6;         // swap-in per DMA
    double gamma = 1.0 / 150e12; // execution per FLOP (layers without a measured time)
    double kappa = 6e-6;         // execution per kernel launch (ditto; also the part
                                 // of a layer's time a slice of it keeps whole)
    double gate = 20e-6;         // compute end -> start of the DMA waiting for it
    double wake = 5e-6;          // DMA end -> start of the compute waiting for it
    double slab_ex = 6e-6;       // per slab on the compute stream, beyond its layers
    std::vector<double> layer_ex;   // measured seconds per layer (< 0: not measured)
};

struct PlanTimes {
    double latency = 0;   // one inference, from an idle start
    double period = 0;    // per inference, back to back, steady state
};

// Storage tier (imagefile.cpp): the planned image in a file, each slab at a
// kFileAlign-aligned offset, read back with direct I/O.
constexpr int64_t kFileAlign = 4096;   // direct-I/O alignment of offsets, sizes, buffers
int64_t image_file_slab_off(const PlanResult &plan, int i);
int image_file_write(const std::string &path, const PlanResult &plan, const uint8_t *image,
                     std::string &err);
// Opens `path` (O_DIRECT when the file system allows it: `direct`), checks
// its header against `plan` and returns the descriptor (-1 on error) and the
// slabs' file offsets.
int image_file_open(const std::string &path, const PlanResult &plan, std::vector<int64_t> &file_off,
                    bool &direct, std::string &err);
// Reads `bytes` rounded up to kFileAlign at `off` into `dst` (kFileAlign
// aligned, room for the rounded size).
int image_file_read(int fd, int64_t off, int64_t bytes, uint8_t *dst, std::string &err);

// Host-only planning (no device calls).
int validate_layers(std::vector<Layer> &layers, int from, std::vector<Slot> &slots,
                    std::string &err);
int prepack_layer(Layer &L, const uint8_t *blob, size_t blob_bytes, std::string &err);
// partition: 0 user blocks, 1 balanced, 2 searched under `cost` (sn_option
// SN_OPT_PARTITION).  `arena_budget` is where the slabs will be placed.
int plan_slabs(const std::vector<Layer> &layers, int n_blocks, int64_t split_budget,
               int64_t arena_budget, int64_t max_slab, int partition, const CostModel &cost,
               PlanResult &out, std::string &err);
void layout_slabs(const std::vector<Layer> &layers, const std::vector<SlabSpec> &specs,
                  PlanResult &out);
int64_t spec_bytes(const std::vector<Layer> &layers, const SlabSpec &s);
int place_slabs(PlanResult &p, int64_t arena_budget, std::string &err);
double layer_flops(const Layer &L);
PlanTimes simulate_plan(const std::vector<Layer> &layers, const PlanResult &placed,
                        const CostModel &cost);
// The partition with the least predicted steady-state time per inference
// (then the least latency) among `seeds` and the searched candidates.
int search_partition(const std::vector<Layer> &layers, int64_t split_budget,
                     int64_t arena_budget, int64_t max_slab, const CostModel &cost,
                     const std::vector<std::vector<SlabSpec>> &seeds,
                     std::vector<SlabSpec> &best, std::string &err);
void assign_slot_offsets(std::vector<Slot> &slots, int64_t &total);
void write_image(const std::vector<Layer> &layers, const PlanResult &p, uint8_t *image);
void choose_kernels(std::vector<Layer> &layers);

}  // namespace sn
