// Step graphs: a hook step captured once and replayed, with the kernel-node
// parameter update the paper uses for dynamic arguments on a fixed path
// (Sec. 4.3, CUDA-graph-safe kernel design; graph-level toggling).
//
// The caller enqueues any sequence of library calls on one stream between
// xmix_graph_begin and xmix_graph_end.  The executor instantiates the
// captured graph and keeps, for every kernel node launched by this library,
// the node handle and a copy of its argument bytes, decoded with the
// argument layout of that kernel (kernels.hpp).  xmix_graph_redirect then
// points every pointer argument that holds one device buffer at another
// (also the pointers inside the batched calls' app descriptors),
// through hipGraphExecKernelNodeSetParams on the affected nodes only: no
// recapture and no re-instantiation.  This is the node-update path; the
// library's own design keeps per-step values in device memory, which needs
// no update at all, and the benchmark compares the two.
//
// Unlike the rest of the library, the executor allocates: host memory for
// its node table and the HIP graph objects, released by xmix_graph_destroy.
#include <string.h>

#include <vector>

#include "../../include/xmix.h"
#include "kernels.hpp"

using namespace xmix;

struct xmix_graph {
    struct Node {
        hipGraphNode_t node;
        hipKernelNodeParams params;   // grid, block, function as captured
        const KernelInfo* info;
        std::vector<uint8_t> bytes;   // current argument values, packed
        std::vector<size_t> offset;   // of each argument in `bytes`
    };
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    std::vector<Node> nodes;
};

namespace {

const std::vector<KernelInfo>& kernel_table() {
    static const std::vector<KernelInfo> table = [] {
        std::vector<KernelInfo> t;
        add_route_kernels(t);
        add_steer_kernels(t);
        add_steer_probe_kernels(t);
        add_probe_kernels(t);
        add_router_kernels(t);
        add_sae_kernels(t);
        add_clamp_kernels(t);
        add_compact_kernels(t);
        return t;
    }();
    return table;
}

const KernelInfo* find_kernel(const void* func) {
    for (const KernelInfo& k : kernel_table())
        if (k.func == func) return &k;
    return nullptr;
}

void release(xmix_graph* g) {
    if (!g) return;
    if (g->exec) (void)hipGraphExecDestroy(g->exec);
    if (g->graph) (void)hipGraphDestroy(g->graph);
    delete g;
}

}  // namespace

extern "C" {

xmix_status xmix_graph_begin(void* stream) {
    if (!stream) return XMIX_E_INVAL;  // the null stream cannot be captured
    const hipError_t e =
        hipStreamBeginCapture(static_cast<hipStream_t>(stream), hipStreamCaptureModeThreadLocal);
    return e == hipSuccess ? XMIX_OK : XMIX_E_LAUNCH;
}

xmix_status xmix_graph_end(void* stream, xmix_graph** out) {
    if (!stream || !out) return XMIX_E_INVAL;
    *out = nullptr;
    xmix_graph* g = new xmix_graph();
    if (hipStreamEndCapture(static_cast<hipStream_t>(stream), &g->graph) != hipSuccess ||
        !g->graph) {
        release(g);
        return XMIX_E_LAUNCH;
    }
    size_t n = 0;
    if (hipGraphGetNodes(g->graph, nullptr, &n) != hipSuccess) {
        release(g);
        return XMIX_E_LAUNCH;
    }
    std::vector<hipGraphNode_t> all(n);
    if (n && hipGraphGetNodes(g->graph, all.data(), &n) != hipSuccess) {
        release(g);
        return XMIX_E_LAUNCH;
    }
    for (hipGraphNode_t node : all) {
        hipGraphNodeType type;
        if (hipGraphNodeGetType(node, &type) != hipSuccess || type != hipGraphNodeTypeKernel)
            continue;
        hipKernelNodeParams p;
        memset(&p, 0, sizeof(p));
        if (hipGraphKernelNodeGetParams(node, &p) != hipSuccess || !p.kernelParams) continue;
        const KernelInfo* info = find_kernel(p.func);
        if (!info) continue;  // not one of this library's kernels
        xmix_graph::Node rec;
        rec.node = node;
        rec.params = p;
        rec.info = info;
        size_t at = 0;
        for (size_t i = 0; i < info->size.size(); ++i) {
            at = (at + 7) / 8 * 8;
            rec.offset.push_back(at);
            at += info->size[i];
        }
        rec.bytes.resize(at);
        for (size_t i = 0; i < info->size.size(); ++i)
            memcpy(rec.bytes.data() + rec.offset[i], p.kernelParams[i], info->size[i]);
        g->nodes.push_back(std::move(rec));
    }
    if (hipGraphInstantiate(&g->exec, g->graph, nullptr, nullptr, 0) != hipSuccess) {
        release(g);
        return XMIX_E_LAUNCH;
    }
    *out = g;
    return XMIX_OK;
}

int32_t xmix_graph_kernel_nodes(const xmix_graph* g) {
    return g ? static_cast<int32_t>(g->nodes.size()) : 0;
}

xmix_status xmix_graph_redirect(xmix_graph* g, const void* from, const void* to,
                                int32_t* n_args) {
    if (n_args) *n_args = 0;
    if (!g || !from || !to) return XMIX_E_INVAL;
    int32_t count = 0;
    std::vector<void*> args;
    for (xmix_graph::Node& rec : g->nodes) {
        bool hit = false;
        for (size_t i = 0; i < rec.info->size.size(); ++i) {
            for (const uint16_t at : rec.info->ptr_at[i]) {  // pointers, also inside structs
                uint8_t* where = rec.bytes.data() + rec.offset[i] + at;
                void* v;
                memcpy(&v, where, sizeof(v));
                if (v != from) continue;
                memcpy(where, &to, sizeof(to));
                hit = true;
                ++count;
            }
        }
        if (!hit) continue;
        args.resize(rec.info->size.size());
        for (size_t i = 0; i < args.size(); ++i) args[i] = rec.bytes.data() + rec.offset[i];
        hipKernelNodeParams p = rec.params;
        p.kernelParams = args.data();
        p.extra = nullptr;
        if (hipGraphExecKernelNodeSetParams(g->exec, rec.node, &p) != hipSuccess)
            return XMIX_E_LAUNCH;
    }
    if (n_args) *n_args = count;
    return XMIX_OK;
}

xmix_status xmix_graph_launch(const xmix_graph* g, void* stream) {
    if (!g || !g->exec) return XMIX_E_INVAL;
    return hipGraphLaunch(g->exec, static_cast<hipStream_t>(stream)) == hipSuccess
               ? XMIX_OK
               : XMIX_E_LAUNCH;
}

void xmix_graph_destroy(xmix_graph* g) { release(g); }

}  // extern "C"
