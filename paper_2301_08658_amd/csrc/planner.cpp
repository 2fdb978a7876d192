// Mesh planner of adaptive tensor parallelism (host code, no GPU).
//
// Search space (Sec. 3.2): every DeviceMesh(d1, d2) with d1 * d2 = N.
// Interconnect (Sec. 3.4): a hierarchical communication matrix, layers
// outermost first, each with a rank count, a per-rank group bandwidth and a
// P2P bandwidth matrix among the ranks of one parent.
// Bandwidths (Sec. 3.5): B1', B2' by Eq. (bwd) with the P2P correction and
// the sharing rule stated in atp.h; B = d / (2 (d - 1)) B' by
// Eq. (allreduce).  Time (Sec. 3.3): Eq. (tcomm).
//
// For one axis and one layer the work is organised per layer-j rank of the
// whole machine ("slot" = (r / D_j), the rank's global index at that layer):
// a first pass marks which slots each axis group touches and groups the
// marks by parent, a second counts for every slot how many groups span the
// layer through it, a third evaluates the bottleneck.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <limits>
#include <vector>

#include "../../include/atp.h"
#include "errors.h"

namespace {

using atp::set_error;

constexpr double kInf = std::numeric_limits<double>::infinity();

struct Hcm {
    int n = 0;                      // layers
    int64_t devices = 1;
    std::vector<int32_t> R;         // ranks per parent
    std::vector<int64_t> D;         // devices per rank of the layer
    std::vector<double> G;          // group bandwidth
    std::vector<const double*> P;   // P2P matrices (may be NULL)

    double p2p(int j, int u, int v) const {
        if (u == v) return 0.0;
        return P[j] ? P[j][(size_t)u * R[j] + v] : G[j];
    }
};

atp_status load_hcm(const atp_hcm_layer* hcm, int32_t n_layers, Hcm* h) {
    if (!hcm) return set_error(ATP_ERR_INVALID_ARGUMENT, "hcm is NULL");
    if (n_layers < 1 || n_layers > ATP_PLAN_MAX_LAYERS)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "n_layers %d outside 1..%d", n_layers,
                         ATP_PLAN_MAX_LAYERS);
    h->n = n_layers;
    h->R.resize(n_layers);
    h->D.resize(n_layers);
    h->G.resize(n_layers);
    h->P.resize(n_layers);
    for (int j = 0; j < n_layers; ++j) {
        const atp_hcm_layer& ly = hcm[j];
        if (ly.ranks < 1)
            return set_error(ATP_ERR_INVALID_ARGUMENT, "layer %d: ranks %d < 1", j, ly.ranks);
        if (!(ly.group_bw > 0.0) || !isfinite(ly.group_bw))
            return set_error(ATP_ERR_INVALID_ARGUMENT, "layer %d: group_bw must be finite and > 0",
                             j);
        h->devices *= ly.ranks;
        if (h->devices > ATP_PLAN_MAX_DEVICES)
            return set_error(ATP_ERR_UNSUPPORTED, "more than %d devices", ATP_PLAN_MAX_DEVICES);
        if (ly.p2p) {
            for (int64_t e = 0; e < (int64_t)ly.ranks * ly.ranks; ++e) {
                const double x = ly.p2p[e];
                if (!(x >= 0.0) || !isfinite(x))
                    return set_error(ATP_ERR_INVALID_ARGUMENT,
                                     "layer %d: p2p entry %lld is negative or not finite", j,
                                     (long long)e);
            }
        }
        h->R[j] = ly.ranks;
        h->G[j] = ly.group_bw;
        h->P[j] = ly.p2p;
    }
    int64_t inner = 1;
    for (int j = n_layers - 1; j >= 0; --j) {
        h->D[j] = inner;
        inner *= h->R[j];
    }
    return ATP_OK;
}

atp_status check_dims(const atp_model_dims* d) {
    if (!d) return set_error(ATP_ERR_INVALID_ARGUMENT, "dims is NULL");
    if (d->layers < 1 || d->batch < 1 || d->seq < 1 || d->hidden < 1 || d->elem_bytes < 1)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "model sizes and elem_bytes must be >= 1");
    return ATP_OK;
}

// Eq. (tcomm); a term whose bandwidth is +inf vanishes, a zero bandwidth
// makes the time infinite.
double tcomm(const atp_model_dims* d, int d1, int d2, double b1, double b2) {
    const double scale = 2.0 * (double)d->layers * (double)d->batch * (double)d->seq *
                         (double)d->elem_bytes / 1e9;
    const double h = (double)d->hidden;
    auto term = [](double num, int dd, double bw) {
        if (isinf(bw)) return 0.0;
        if (bw <= 0.0) return kInf;
        return num / ((double)dd * bw);
    };
    return scale * (term(7.0 * h, d1, b2) + term(2.0 * h, d2, b1));
}

// B' of one axis (Eq. (bwd)).  Groups: axis 1 -> devices with equal i2
// (members i1 * d2 + i2), axis 2 -> equal i1 (members i1 * d2 + i2).
double axis_bandwidth(const Hcm& h, int d1, int d2, int axis) {
    const int n_groups = axis == 1 ? d2 : d1;
    const int g_size = axis == 1 ? d1 : d2;
    auto member = [&](int g, int k) -> int64_t {
        return axis == 1 ? (int64_t)k * d2 + g : (int64_t)g * d2 + k;
    };
    double best = kInf;
    for (int j = 0; j < h.n; ++j) {
        const int64_t slots = h.devices / h.D[j];   // layer-j ranks of the machine
        const int R = h.R[j];
        // slot of device r = r / D_j; parent = slot / R; rank in parent = slot % R
        std::vector<int32_t> through(slots, 0);       // spanning groups per slot
        std::vector<std::vector<int64_t>> spans;      // per (group, parent) with > 1 rank
        std::vector<int64_t> tmp;
        for (int g = 0; g < n_groups; ++g) {
            tmp.clear();
            for (int k = 0; k < g_size; ++k) tmp.push_back(member(g, k) / h.D[j]);
            std::sort(tmp.begin(), tmp.end());
            tmp.erase(std::unique(tmp.begin(), tmp.end()), tmp.end());
            // split the touched slots by parent
            size_t a = 0;
            while (a < tmp.size()) {
                size_t b = a;
                while (b < tmp.size() && tmp[b] / R == tmp[a] / R) ++b;
                if (b - a > 1) {
                    spans.emplace_back(tmp.begin() + a, tmp.begin() + b);
                    for (size_t q = a; q < b; ++q) ++through[tmp[q]];
                }
                a = b;
            }
        }
        for (const std::vector<int64_t>& sp : spans) {
            for (int64_t su : sp) {
                const int u = (int)(su % R);
                double sum = 0.0;
                for (int64_t sv : sp) sum += h.p2p(j, u, (int)(sv % R));
                const double bw = std::min(h.G[j], sum) / (double)through[su];
                best = std::min(best, bw);
            }
        }
    }
    return best;   // every group of >= 2 devices spans some layer, so this is finite
}

void mesh_cost(const Hcm& h, const atp_model_dims* dims, int d1, int d2, atp_mesh_cost* c) {
    c->d1 = d1;
    c->d2 = d2;
    c->b1_eff = d1 > 1 ? axis_bandwidth(h, d1, d2, 1) : 0.0;
    c->b2_eff = d2 > 1 ? axis_bandwidth(h, d1, d2, 2) : 0.0;
    c->b1 = d1 > 1 ? (double)d1 / (2.0 * (d1 - 1)) * c->b1_eff : kInf;
    c->b2 = d2 > 1 ? (double)d2 / (2.0 * (d2 - 1)) * c->b2_eff : kInf;
    c->t_comm = tcomm(dims, d1, d2, c->b1, c->b2);
}

}  // namespace

extern "C" {

atp_status atp_tcomm(const atp_model_dims* dims, int32_t d1, int32_t d2, double b1, double b2,
                     double* t_out) {
    if (!t_out) return set_error(ATP_ERR_INVALID_ARGUMENT, "t_out is NULL");
    atp_status s = check_dims(dims);
    if (s != ATP_OK) return s;
    if (d1 < 1 || d2 < 1) return set_error(ATP_ERR_INVALID_ARGUMENT, "mesh sizes must be >= 1");
    if (!(b1 > 0.0) || !(b2 > 0.0))
        return set_error(ATP_ERR_INVALID_ARGUMENT, "bandwidths must be > 0 (+inf allowed)");
    *t_out = tcomm(dims, d1, d2, b1, b2);
    return ATP_OK;
}

atp_status atp_hcm_mesh_cost(const atp_hcm_layer* hcm, int32_t n_layers,
                             const atp_model_dims* dims, int32_t d1, int32_t d2,
                             atp_mesh_cost* out) {
    if (!out) return set_error(ATP_ERR_INVALID_ARGUMENT, "out is NULL");
    Hcm h;
    atp_status s = load_hcm(hcm, n_layers, &h);
    if (s != ATP_OK) return s;
    s = check_dims(dims);
    if (s != ATP_OK) return s;
    if (d1 < 1 || d2 < 1) return set_error(ATP_ERR_INVALID_ARGUMENT, "mesh sizes must be >= 1");
    if ((int64_t)d1 * d2 != h.devices)
        return set_error(ATP_ERR_SHAPE, "DeviceMesh(%d, %d) does not cover the HCM's %lld devices",
                         d1, d2, (long long)h.devices);
    mesh_cost(h, dims, d1, d2, out);
    return ATP_OK;
}

atp_status atp_plan_mesh(const atp_hcm_layer* hcm, int32_t n_layers, const atp_model_dims* dims,
                         atp_mesh_cost* best, atp_mesh_cost* costs, int32_t max_costs,
                         int32_t* n_meshes) {
    if (!best) return set_error(ATP_ERR_INVALID_ARGUMENT, "best is NULL");
    Hcm h;
    atp_status s = load_hcm(hcm, n_layers, &h);
    if (s != ATP_OK) return s;
    s = check_dims(dims);
    if (s != ATP_OK) return s;
    const int N = (int)h.devices;
    std::vector<int> d1s;
    for (int d1 = N; d1 >= 1; --d1)
        if (N % d1 == 0) d1s.push_back(d1);
    const int n = (int)d1s.size();
    if (costs && max_costs < n)
        return set_error(ATP_ERR_INVALID_ARGUMENT, "costs holds %d entries, %d meshes", max_costs,
                         n);
    atp_mesh_cost pick;
    memset(&pick, 0, sizeof pick);
    for (int q = 0; q < n; ++q) {
        atp_mesh_cost c;
        mesh_cost(h, dims, d1s[q], N / d1s[q], &c);
        if (costs) costs[q] = c;
        if (q == 0 || c.t_comm < pick.t_comm) pick = c;
    }
    *best = pick;
    if (n_meshes) *n_meshes = n;
    return ATP_OK;
}

}  // extern "C"
