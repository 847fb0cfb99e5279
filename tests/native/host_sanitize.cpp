// Host-only driver for the stage library's planner (stage_plan_offload) and allocation scheduler
// (stage_allocate), built with the address and undefined-behaviour sanitizers by
// tests/test_host_sanitizers.py.  Reads one instance per line on stdin and prints the library's
// answer on one line, so the test can compare it with the oracle:
//   plan  mem_left kv_per_token mha_bytes mlp_bytes mha_cost mlp_cost mha_free mlp_free n_stage
//     -> rc n capacity tokens:alpha:beta ...
//   alloc n_layers mha_bytes mlp_bytes comm n_devices (mem comp load_mha load_mlp) x n_devices
//     -> rc n_stage t_total first:assigned:offloaded:mha_only:mlp_only ...
// Every instance is asked twice where the API allows a capacity: first with cap = 0 (count only),
// then with an array of exactly the returned count, so both paths run under the sanitizers.
#include <cstdint>
#include <cstdio>
#include <iostream>
#include <sstream>
#include <string>
#include <vector>

#include "stage.h"
#include "stage_alloc.h"
#include "stage_planner.h"

static void run_plan(std::istringstream &in) {
    stage_plan_input p{};
    long long v[9];
    for (long long &x : v) in >> x;
    p.mem_left = v[0]; p.kv_bytes_per_token = v[1]; p.mha_bytes = v[2]; p.mlp_bytes = v[3];
    p.mha_cost = v[4]; p.mlp_cost = v[5];
    p.mha_free = (int32_t)v[6]; p.mlp_free = (int32_t)v[7]; p.n_stage = (int32_t)v[8];
    int32_t n = -1;
    int64_t cap = -1;
    int rc = stage_plan_offload(&p, nullptr, 0, &n, &cap);
    if (rc != STAGE_OK) {
        std::printf("%d\n", rc);
        return;
    }
    std::vector<stage_plan_step> steps((size_t)n);
    rc = stage_plan_offload(&p, steps.data(), n, &n, &cap);
    std::printf("%d %d %lld", rc, n, (long long)cap);
    for (const stage_plan_step &s : steps) std::printf(" %lld:%d:%d", (long long)s.tokens, s.alpha, s.beta);
    std::printf("\n");
}

static void run_alloc(std::istringstream &in) {
    stage_alloc_input a{};
    long long n_layers, mha, mlp, comm, n_dev;
    in >> n_layers >> mha >> mlp >> comm >> n_dev;
    std::vector<stage_alloc_device> devs((size_t)(n_dev > 0 ? n_dev : 0));
    for (stage_alloc_device &d : devs) {
        long long m, c, la, lm;
        in >> m >> c >> la >> lm;
        d.mem_bytes = m; d.comp_layer = c; d.load_mha = la; d.load_mlp = lm;
    }
    a.n_layers = (int32_t)n_layers; a.mha_bytes = mha; a.mlp_bytes = mlp; a.comm = comm;
    a.n_devices = (int32_t)n_dev;
    a.devices = devs.empty() ? nullptr : devs.data();
    std::vector<stage_alloc_plan> out(devs.size());
    int32_t n_stage = -1;
    int64_t t = -1;
    const int rc = stage_allocate(&a, out.empty() ? nullptr : out.data(), &n_stage, &t);
    if (rc != STAGE_OK) {
        std::printf("%d\n", rc);
        return;
    }
    std::printf("%d %d %lld", rc, n_stage, (long long)t);
    for (const stage_alloc_plan &p : out)
        std::printf(" %d:%d:%d:%d:%d", p.first_layer, p.assigned, p.offloaded, p.mha_only, p.mlp_only);
    std::printf("\n");
}

int main() {
    std::string line;
    while (std::getline(std::cin, line)) {
        std::istringstream in(line);
        std::string kind;
        in >> kind;
        if (kind == "plan") run_plan(in);
        else if (kind == "alloc") run_alloc(in);
        else if (!kind.empty()) std::printf("? %s\n", kind.c_str());
    }
    return 0;
}
