// Fine-grained allocation scheduler (Section III-D, Alg. 1; cost model Eq. (1), overlap window
// Eq. (2), dynamic program Eqs. (3)-(4)).  Implements include/stage_alloc.h.
#include <algorithm>
#include <cstdint>
#include <limits>
#include <vector>

#include "stage.h"
#include "stage_alloc.h"

namespace {

constexpr int64_t kMaxTime = int64_t(1) << 40;  // keeps every sum below 2^62
constexpr int64_t kInf = std::numeric_limits<int64_t>::max();

struct Work {
    int D = 0, L = 0;
    int64_t l_size = 0, mha_bytes = 0, mlp_bytes = 0, comm = 0;
    std::vector<int64_t> cap, rem, comp, load_a, load_m;
};

struct Candidate {
    int s = 0;
    int64_t t_total = kInf;
    std::vector<int> k, whole, mha_only, mlp_only;
};

int64_t load_layer(const Work &w, int i) { return w.load_a[i] + w.load_m[i]; }

// Eq. (2) before offloading: own retained layers, every other device's layers, the hops.
std::vector<int64_t> idle_windows(const Work &w) {
    int64_t all = 0;
    for (int i = 0; i < w.D; ++i) all += w.cap[i] * w.comp[i];
    std::vector<int64_t> idle(w.D);
    for (int i = 0; i < w.D; ++i) idle[i] = all + w.D * w.comm;  // C_i*comp_i + sum_{i' != i} C_i'*comp_i'
    return idle;
}

// Eqs. (3)-(4): F(l, i), the least uncovered loading delay once l of the left layers are spread
// over devices 0..i as offloaded layers; returns each device's share.
std::vector<int> stage_dp(const Work &w, int left, const std::vector<int64_t> &idle) {
    const int D = w.D;
    std::vector<std::vector<int64_t>> F(D, std::vector<int64_t>(left + 1, kInf));
    std::vector<std::vector<int>> P(D, std::vector<int>(left + 1, 0));
    for (int l = 0; l <= left; ++l) {
        F[0][l] = std::max<int64_t>(0, l * load_layer(w, 0) - idle[0]);
        P[0][l] = l;
    }
    for (int i = 1; i < D; ++i) {
        F[i][0] = 0;
        for (int l = 1; l <= left; ++l)
            for (int k = 0; k <= l; ++k) {
                const int64_t cur = std::max<int64_t>(0, F[i - 1][l - k] + k * load_layer(w, i) - idle[i]);
                if (cur <= F[i][l]) {
                    F[i][l] = cur;
                    P[i][l] = k;
                }
            }
    }
    std::vector<int> k(D, 0);
    int l = left;
    for (int i = D - 1; i >= 1; --i) {
        k[i] = P[i][l];
        l -= k[i];
    }
    k[0] = l;
    return k;
}

int64_t device_load(const Work &w, int i, int whole, int mha_only, int mlp_only) {
    return whole * load_layer(w, i) + mha_only * w.load_a[i] + mlp_only * w.load_m[i];
}

// Eq. (1) under a candidate plan with s stages per device.
int64_t t_total(const Work &w, const Candidate &c) {
    std::vector<int64_t> comp_dev(w.D);
    int64_t comp_all = 0;
    for (int i = 0; i < w.D; ++i) {
        comp_dev[i] = (w.cap[i] + c.k[i]) * w.comp[i];
        comp_all += comp_dev[i];
    }
    const int64_t hops = (int64_t)w.D * w.comm;
    int64_t uncover = 0;
    for (int i = 0; i < w.D; ++i) {
        const int64_t load = device_load(w, i, c.whole[i], c.mha_only[i], c.mlp_only[i]);
        const int64_t window = w.cap[i] * w.comp[i] + (comp_all - comp_dev[i]) + hops;
        uncover = std::max(uncover, std::max<int64_t>(0, load - window));
    }
    return comp_all + (int64_t)c.s * hops + uncover;
}

// Block-level refinement of the bottleneck device until it cannot improve.
void refine(const Work &w, Candidate &c) {
    std::vector<int64_t> rem = w.rem, T(w.D);
    for (int i = 0; i < w.D; ++i) T[i] = device_load(w, i, c.whole[i], 0, 0);
    for (;;) {
        int top = 0;
        for (int i = 1; i < w.D; ++i)
            if (T[i] > T[top]) top = i;
        if (c.whole[top] < 1) return;
        if (rem[top] >= w.mlp_bytes) {          // keep the MLP block: MHA-only offloading
            rem[top] -= w.mlp_bytes;
            c.whole[top]--;
            c.mha_only[top]++;
            T[top] -= w.load_m[top];
        } else if (rem[top] >= w.mha_bytes) {   // keep the MHA block: MLP-only offloading
            rem[top] -= w.mha_bytes;
            c.whole[top]--;
            c.mlp_only[top]++;
            T[top] -= w.load_a[top];
        } else {
            return;
        }
    }
}

}  // namespace

extern "C" int stage_allocate(const stage_alloc_input *in, stage_alloc_plan *out, int32_t *n_stage,
                              int64_t *t_total_out) {
    if (!in || !out || !n_stage || !t_total_out || !in->devices) return STAGE_EINVAL;
    const stage_alloc_input &p = *in;
    if (p.n_layers < 1 || p.n_layers > STAGE_ALLOC_MAX_LAYERS || p.n_devices < 1 ||
        p.n_devices > STAGE_ALLOC_MAX_DEVICES || p.mha_bytes <= 0 || p.mlp_bytes <= 0 ||
        p.mha_bytes > (int64_t(1) << 52) || p.mlp_bytes > (int64_t(1) << 52) || p.comm < 0 || p.comm > kMaxTime)
        return STAGE_EINVAL;
    Work w;
    w.D = p.n_devices;
    w.L = p.n_layers;
    w.mha_bytes = p.mha_bytes;
    w.mlp_bytes = p.mlp_bytes;
    w.l_size = p.mha_bytes + p.mlp_bytes;
    w.comm = p.comm;
    int64_t cap_sum = 0;
    for (int i = 0; i < w.D; ++i) {
        const stage_alloc_device &d = p.devices[i];
        if (d.mem_bytes < 0 || d.comp_layer < 0 || d.comp_layer > kMaxTime || d.load_mha <= 0 ||
            d.load_mha > kMaxTime || d.load_mlp <= 0 || d.load_mlp > kMaxTime)
            return STAGE_EINVAL;
        const int64_t cap = std::min<int64_t>(d.mem_bytes / w.l_size, STAGE_ALLOC_MAX_LAYERS);
        w.cap.push_back(cap);
        w.rem.push_back(d.mem_bytes - cap * w.l_size);
        w.comp.push_back(d.comp_layer);
        w.load_a.push_back(d.load_mha);
        w.load_m.push_back(d.load_mlp);
        cap_sum += cap;
    }

    const int64_t left = w.L - cap_sum;
    Candidate best;
    if (left <= 0) {  // everything fits: layers in order up to capacity, no offloading
        best.s = 1;
        best.k.assign(w.D, 0);
        best.whole = best.mha_only = best.mlp_only = best.k;
        int64_t need = w.L;
        std::vector<int64_t> cap = w.cap;
        for (int i = 0; i < w.D; ++i) {
            w.cap[i] = std::min(cap[i], need);
            need -= w.cap[i];
        }
        best.t_total = t_total(w, best);
    } else {
        const int s_max = (int)std::min<int64_t>(std::max<int64_t>(2, left), (w.L + w.D - 1) / w.D);
        const std::vector<int64_t> idle = idle_windows(w);
        const std::vector<int> k = stage_dp(w, (int)left, idle);  // the windows do not depend on s
        for (int s = 2; s <= s_max; ++s) {
            bool feasible = true;
            for (int i = 0; i < w.D; ++i)
                if (w.cap[i] + k[i] > (int64_t)s * w.cap[i]) feasible = false;
            if (!feasible) continue;
            Candidate c;
            c.s = s;
            c.k = k;
            c.whole = k;
            c.mha_only.assign(w.D, 0);
            c.mlp_only.assign(w.D, 0);
            refine(w, c);
            c.t_total = t_total(w, c);
            if (c.t_total < best.t_total) best = c;
        }
        if (best.t_total == kInf) return STAGE_ERANGE;
    }
    int first = 0;
    for (int i = 0; i < w.D; ++i) {
        stage_alloc_plan &o = out[i];
        o.first_layer = first;
        o.assigned = (int32_t)(w.cap[i] + best.k[i]);
        o.offloaded = best.k[i];
        o.mha_only = best.mha_only[i];
        o.mlp_only = best.mlp_only[i];
        first += o.assigned;
    }
    *n_stage = best.s;
    *t_total_out = best.t_total;
    return STAGE_OK;
}
