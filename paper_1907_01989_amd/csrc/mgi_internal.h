// Internal data structures of the mgi engine (host side).
//
// Activation storage ("C8 layout"): a tensor (n, h, w, c) is split into
// S = ceil(c / 8) slices of 8 channels; slice s of all n*h*w pixels is stored
// contiguously, pixel-major, 8 fp16 values (16 bytes) per pixel:
//     element (n, y, x, ch) at  ((ch / 8) * M + (n * h + y) * w + x) * 8 + ch % 8
// with M = n * h * w.  Channels c..8S-1 of the last slice are kept at zero.
// This is the channel-sliced layout of the paper (Sec. 4, PHWC4) widened to
// 8 channels so that one lane moves 16 bytes and 8 neighbouring lanes fill a
// 128-byte line; with n = 1 it is exactly PHWC8.
#pragma once

#include <cstddef>
#include <cstdint>
#include <exception>
#include <new>
#include <string>
#include <vector>

#include "../../include/mgi.h"

// Every extern "C" entry point runs its body inside MGI_ABI_TRY /
// MGI_ABI_CATCH(name): no C++ exception crosses the C boundary; an allocation
// failure becomes MGI_ERR_OOM_HOST and anything else MGI_ERR_INTERNAL, with
// the message left in mgi_last_error().
#define MGI_ABI_TRY try {
#define MGI_ABI_CATCH(name)                                                               \
    }                                                                                     \
    catch (const std::bad_alloc &) {                                                      \
        return ::mgi::fail(MGI_ERR_OOM_HOST, std::string(name) + ": out of host memory"); \
    }                                                                                     \
    catch (const std::exception &e) {                                                     \
        return ::mgi::fail(MGI_ERR_INTERNAL, std::string(name) + ": " + e.what());        \
    }                                                                                     \
    catch (...) {                                                                         \
        return ::mgi::fail(MGI_ERR_INTERNAL, std::string(name) + ": unknown exception");  \
    }

namespace mgi {

enum class OpKind {
    Input, Conv2d, Depthwise, Add, Activation, GlobalAvgPool, FC, Softmax, Concat,
    ResizeBilinear, Argmax, Pad
};

struct Shape {
    int n = 0, h = 0, w = 0, c = 0;
    size_t pixels() const { return (size_t)n * h * w; }
    size_t elems() const { return pixels() * c; }
};

// One graph operator; its output is tensor id == its index in Graph::ops.
struct GOp {
    OpKind kind;
    std::vector<int> in;
    Shape out;
    mgi_conv_desc conv{};       // Conv2d / Depthwise
    int act = MGI_ACT_NONE;     // Conv2d / Depthwise / Add / Activation
    int in_dtype = MGI_DTYPE_FP32;  // Input
    int oh = 0, ow = 0, align_corners = 1;  // ResizeBilinear
    int cout = 0;               // FC
    int pads[4] = {0, 0, 0, 0}; // Pad: top, bottom, left, right
    std::vector<float> w, b;    // weights as given (OHWI / CHW / COUT x CIN), bias
};

}  // namespace mgi

struct mgi_graph {
    std::vector<mgi::GOp> ops;
    std::vector<int> outputs;
    std::vector<int> inputs;  // tensor ids of Input ops, in declaration order
};

namespace mgi {

// Storage classes of materialised tensors.
enum class Layout { C8, F32, I32, NHWC_IN };
enum class Loc { Arena, Input, Output };

struct Buf {
    Layout layout = Layout::C8;
    Shape shape;
    size_t bytes = 0;
    Loc loc = Loc::Arena;
    int index = -1;          // input / output index for Loc::Input / Loc::Output
    size_t offset = 0;       // arena offset for Loc::Arena
    int producer = -1;       // node index (-1: graph input)
    int last_use = -1;       // last node index that reads it (-1: none)
    int graph_tensor = -1;   // graph tensor id it holds (-1: internal)
    bool dead = false;       // no longer produced or read (fused away); not planned
    int in_dtype = MGI_DTYPE_FP32;  // element type of a NHWC_IN buffer
};

enum class NodeKind {
    Ingest, Stem, Gemm, Depthwise, Add, Act, Gap, FC, Softmax, Concat, Resize, Argmax,
    ResizeArgmax, Export, Pad, DwPw, PwDw, StemDw, GemmPool, FcSoftmax, Irb
};

// Tile shape of the MFMA GEMM (pointwise, implicit-GEMM convolution, FC).
// pipe = true selects the pipelined pointwise kernel with bm x bn tiles;
// slab = true the weight-slab pointwise kernel with (4 * wm) x bn tiles and
// pf K steps of activation prefetch; otherwise the LDS-staged kernel with
// bm x bn tiles.
struct GemmTile {
    int bm = 64, bn = 64;
    bool pipe = false;
    bool slab = false;
    int wm = 32, pf = 1;
    int ks = 4;             // pipe: K slices per ring stage (4, or 8 for 64 x 64 tiles)
};

struct Node {
    NodeKind kind;
    const char *kname = "";
    int op = -1;            // heavy graph op (first absorbed)
    int out_tensor = -1;    // graph tensor represented by the output
    int n_fused = 1;        // graph ops absorbed
    std::vector<int> in;    // buffer ids
    int out = -1;           // buffer id
    int residual = -1;      // buffer id (Gemm / Stem epilogue), -1 = none
    int act1 = MGI_ACT_NONE, act2 = MGI_ACT_NONE;
    // weights in the packed blob
    size_t w_off = 0, w_bytes = 0, b_off = 0, b_bytes = 0;
    // GEMM geometry
    int ksl = 0;            // K slices (8 wide) before padding
    int ksp = 0;            // K slices padded to a multiple of 4
    int nb16 = 0;           // output channel blocks of 16
    bool taps = false;      // implicit GEMM over a kh x kw window
    GemmTile tile;
    mgi_conv_desc conv{};
    int align_corners = 1;
    int dw_rows = 0;        // depthwise 3x3: output rows per thread (0 = kernel default)
    // DwPw / PwDw: the absorbed depthwise op (the pointwise input's producer,
    // or the pointwise output's consumer), its window, activation and packed
    // taps
    int dw_op = -1;
    mgi_conv_desc dw_conv{};
    int dw_act = MGI_ACT_NONE;
    size_t dw_w_off = 0, dw_b_off = 0;
    Shape dw_in, dw_out;    // PwDw / StemDw / GemmPool: shapes of the intermediate tensor (the first
                            // op's output) and of the node's output
    // kernel configurations the autotuner may choose from (index 0 = the
    // finalize-time choice); `cfg` is the one in use
    // PwDw / StemDw / GemmPool: the first op's output kept as a planned scratch tensor,
    // so that the node can also run as the two separate kernels (split);
    // whether the fused kernel is the default configuration
    int scratch = -1;
    bool split = false;
    bool fused_default = true;
    bool irb_default = false;   // Irb: the block kernel is the default configuration
    int pwdw_cfg = 0;       // PwDw / StemDw: configuration of the fused kernel (pwdw_configs,
                            // stemdw_configs)
    size_t cnt_off = 0;     // FcSoftmax: its row-tile arrival counters in the workspace's
                            // state region
    // Irb (a PwDw node that also runs the pointwise projection reading its
    // output): the projection's graph op, packed weights, GEMM geometry and
    // epilogue (residual in `residual`), the depthwise output kept as a
    // second planned scratch tensor (`scratch2`) for the split forms, and the
    // projection's GEMM tile in those forms
    int pj_op = -1;
    size_t pj_w_off = 0, pj_b_off = 0;
    int pj_ksl = 0, pj_ksp = 0, pj_nb16 = 0;
    int pj_act1 = MGI_ACT_NONE, pj_act2 = MGI_ACT_NONE;
    int scratch2 = -1;
    GemmTile pj_tile;
    int mode = 0;           // Irb: 0 the block kernel (pwdw_cfg: its configuration), 1 the fused
                            // pointwise -> depthwise kernel (pwdw_cfg) then the projection GEMM,
                            // 2 three kernels (expansion GEMM `tile`, depthwise, projection GEMM)
    struct Config {
        GemmTile tile;
        int dw_rows = 0;
        std::string name;
        bool split = false;
        int pwdw_cfg = 0;
        int mode = 0;
    };
    std::vector<Config> cfgs;
    int cfg = 0;
    void apply(int c) {
        cfg = c;
        tile = cfgs[c].tile;
        dw_rows = cfgs[c].dw_rows;
        split = cfgs[c].split;
        pwdw_cfg = cfgs[c].pwdw_cfg;
        mode = cfgs[c].mode;
    }
};

}  // namespace mgi

struct mgi_plan {
    std::vector<mgi::Node> nodes;
    std::vector<mgi::Buf> bufs;
    std::vector<int> input_bufs;   // graph input i -> buffer id
    std::vector<int> output_bufs;  // graph output i -> buffer id
    std::vector<int> output_tensor;
    std::vector<mgi::Shape> input_shapes, output_shapes;
    std::vector<int> input_dtypes, output_dtypes;
    std::vector<uint8_t> weights;  // packed host copy (released after bind)
    size_t weight_bytes = 0;
    size_t zero_off = 0;           // offset of a zeroed 256-byte block in the weight blob
    size_t workspace_bytes = 0;
    // state region of the workspace, past the arena (never shared by the
    // planner): zeroed by mgi_plan_bind; kernels that keep counters there leave
    // them at zero when they finish
    size_t state_off = 0, state_bytes = 0;
    size_t mem_naive = 0, mem_planned = 0;
    int n_objects = 0;
    mgi_options opt{};
    void *dev_ws = nullptr;
    void *dev_w = nullptr;
    bool bound = false;
    std::vector<void *> last_outputs;  // output pointers of the latest run
    void *last_ws = nullptr;           // workspace base of the latest run
    void *graph = nullptr;             // hipGraph_t of the captured launch list
    void *graph_exec = nullptr;        // hipGraphExec_t
    std::vector<void *> graph_outputs; // output pointers baked into the graph
    ~mgi_plan();
};

namespace mgi {

// error reporting (thread-local last error)
mgi_status fail(mgi_status s, const std::string &msg);

// planner (Sec. 5).  Tensors are given by size and lifetime [first, last]
// in node order (last = -1: never consumed).
struct PlanResult {
    std::vector<int> object_of;
    std::vector<size_t> object_size;
};
PlanResult plan_naive(const std::vector<size_t> &sizes);
PlanResult plan_greedy(const std::vector<size_t> &sizes, const std::vector<int> &first,
                       const std::vector<int> &last);
PlanResult plan_mcfp(const std::vector<size_t> &sizes, const std::vector<int> &first,
                     const std::vector<int> &last);

// finalize steps
mgi_status build_plan(const mgi_graph &g, const mgi_options &o, mgi_plan &p);

namespace kern {
struct StemDwParams;
}
// shape fields of the fused stem -> depthwise kernel's parameters for a
// StemDw node (pointers and storage type left to the caller)
void stemdw_shape(const mgi_plan &p, const Node &nd, kern::StemDwParams &q);

}  // namespace mgi
