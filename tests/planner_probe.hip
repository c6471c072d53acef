// Host-side probe of the dispatch planners (test infrastructure): reads one
// call per line from stdin and prints the plan the library would use, so
// that the CPU tests can check the plans' invariants and the documented
// choices without a GPU.  It includes the dispatch source itself, so the
// functions it calls are the library's own.
//
//   wide <fmt> <epi> <M> <N1> <K1> [<N2> <K2> ...]  -> plan_splits (large M)
//   stream <fmt> <M> <N1> <K1> [...]                 -> stream_plan (few rows)
//
// Output, one line per input: "wide ext S1 ps1 S2 ps2 ..." (layers in the
// order the library launches them: longest reduction first) or
// "stream rw kw mx S1 pb1 S2 pb2 ...".
#include "../paper_2607_08526_amd/csrc/qlinear.hip"

#include <cstdio>
#include <iostream>
#include <sstream>
#include <string>

int main()
{
    using namespace qlk;
    std::string line;
    while (std::getline(std::cin, line)) {
        std::istringstream in(line);
        std::string kind;
        int fmt = 0, epi = 0, M = 0;
        in >> kind >> fmt;
        if (kind == "wide")
            in >> epi;
        in >> M;
        LinDesc d[QL_MAX_GROUP]{};
        int n = 0, N, K;
        while (n < QL_MAX_GROUP && in >> N >> K) {
            LinDesc &x = d[n++];
            x.M = M;
            x.N = N;
            x.K = K;
            x.tiles_m = (M + wide_tile_bm() - 1) / wide_tile_bm();
            x.tiles_n = (N + wide_tile_bn() - 1) / wide_tile_bn();
            x.ksplit = 1;
            x.psteps = K / 64;
            if (epi)
                x.ep.bias = reinterpret_cast<const float *>(16);
        }
        if (kind == "wide") {
            std::stable_sort(d, d + n, [](const LinDesc &a, const LinDesc &b) { return a.K > b.K; });
            const SplitPlan pl = plan_splits(fmt, d, n);
            std::printf("wide %d", pl.ext ? 1 : 0);
            for (int i = 0; i < n; ++i)
                std::printf(" %d %d %d %d", d[i].K, d[i].tiles_m * d[i].tiles_n, pl.S[i], pl.psteps[i]);
        } else {
            int S[QL_MAX_GROUP], P[QL_MAX_GROUP];
            const StreamPlan sp = stream_plan(fmt, d, n, device_cus(), S, P);
            std::printf("stream %d %d %d", sp.rw, sp.kw, sp.mx);
            for (int i = 0; i < n; ++i)
                std::printf(" %d %d %d", d[i].K, S[i], P[i]);
        }
        std::printf("\n");
    }
    return 0;
}
