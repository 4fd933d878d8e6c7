// Test driver of the library's host-side scheduler for the sanitizer build
// (AddressSanitizer and UndefinedBehaviorSanitizer on the host code of
// api.hip): builds each network of an input file with psw_net_create, queries
// its sizes and parameter offsets, writes the dry-run plan (psw_net_plan) of
// steps 0..T-1 and exercises the argument checks that need no device.  No
// HIP call is made.  Test infrastructure only.
//
// Input: int32 count of nets, then per net: int32 n_ops, batch, c0, h0, w0,
// n_stages, prec, T; int32 desc[9*n_ops], stage_end[n_stages],
// ring_depth[n_stages], staleness[T*n_stages].
// Output (text): per net one line "sizes <stage params...> <ring> <params>
// <bn> <arena>", one line per step "plan t <n> (op what stage version)*",
// and one line "checks ok".
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <vector>

#include "../../include/psw.h"

static bool rd(FILE* f, void* p, size_t bytes) { return fread(p, 1, bytes, f) == bytes; }

int main(int argc, char** argv)
{
    if (argc != 2) return 2;
    FILE* f = fopen(argv[1], "rb");
    if (!f) return 2;
    int32_t nets = 0;
    if (!rd(f, &nets, 4)) return 2;
    for (int k = 0; k < nets; ++k) {
        int32_t h[8];
        if (!rd(f, h, sizeof(h))) return 2;
        const int n_ops = h[0], batch = h[1], c0 = h[2], h0 = h[3], w0 = h[4], S = h[5], prec = h[6], T = h[7];
        std::vector<psw_layer> ops(n_ops);
        std::vector<int32_t> se(S), rd_(S), st((size_t)T * S);
        if (!rd(f, ops.data(), sizeof(psw_layer) * n_ops) || !rd(f, se.data(), 4 * S) || !rd(f, rd_.data(), 4 * S) ||
            !rd(f, st.data(), 4 * st.size()))
            return 2;
        psw_net* net = nullptr;
        if (psw_net_create(ops.data(), n_ops, batch, c0, h0, w0, se.data(), S, rd_.data(), prec, &net) != PSW_OK) {
            fprintf(stderr, "net %d: %s\n", k, psw_last_error());
            return 3;
        }
        std::vector<int64_t> sp(S);
        int64_t ring = 0, np = 0, bn = 0, arena = 0;
        if (psw_net_sizes(net, sp.data(), &ring, &np, &bn, &arena) != PSW_OK) return 4;
        printf("sizes");
        for (int s = 0; s < S; ++s) printf(" %lld", (long long)sp[s]);
        printf(" %lld %lld %lld %lld\n", (long long)ring, (long long)np, (long long)bn, (long long)arena);
        for (int i = 0; i < n_ops; ++i) {
            int stage = -1;
            int64_t off = -1, cnt = -1;
            if (psw_net_param_offset(net, i, &stage, &off, &cnt) != PSW_OK) return 5;
        }
        std::vector<psw_launch> plan(4096);
        for (int t = 0; t < T; ++t) {
            int n = 0;
            if (psw_net_plan(net, t, st.data() + (size_t)t * S, plan.data(), (int)plan.size(), &n) != PSW_OK) return 6;
            printf("plan %d %d", t, n);
            for (int i = 0; i < n && i < (int)plan.size(); ++i)
                printf(" %d %d %d %lld", plan[i].op, plan[i].what, plan[i].stage, (long long)plan[i].version);
            printf("\n");
        }
        // argument checks that stay on the host
        std::vector<int32_t> bad(st.begin(), st.begin() + S);
        bad[0] = rd_[0];  // staleness == ring depth
        int n = 0;
        if (psw_net_plan(net, 5, bad.data(), plan.data(), 4, &n) != PSW_ERR_STALENESS) return 7;
        if (psw_net_param_offset(net, n_ops, nullptr, nullptr, nullptr) != PSW_ERR_SHAPE) return 8;
        float* ptr = nullptr;
        if (psw_net_tensor(net, 1, 0, &ptr, nullptr) != PSW_ERR_STATE) return 9;   // not bound
        if (psw_net_slot(net, 0, 0, &ptr) != PSW_ERR_STATE) return 10;            // not bound
        if (psw_net_set_weight_stashing(net, 1) != PSW_OK || psw_net_set_step(net, 3) != PSW_OK) return 11;
        if (psw_net_profile_replay(net, 0) != PSW_ERR_SHAPE) return 12;
        psw_net_destroy(net);
        // a PPV that does not end at the last operation is refused
        std::vector<int32_t> se2(se);
        se2[S - 1] = n_ops - 1;
        psw_net* net2 = nullptr;
        if (psw_net_create(ops.data(), n_ops, batch, c0, h0, w0, se2.data(), S, rd_.data(), prec, &net2) == PSW_OK)
            return 13;
        psw_net_destroy(net2);
        printf("checks ok\n");
    }
    fclose(f);
    return 0;
}
