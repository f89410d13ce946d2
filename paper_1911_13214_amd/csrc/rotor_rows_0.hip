// Row edges with 0 to 3 low splits (see rotor_rows.h).
#include "rotor_rows.h"

namespace rotor {

void launch_edge_row_0(int a, dim3 grid, hipStream_t stream, const Tables &tb, int delta, int finish, const Work &w)
{
    launch_edge_row_range<0, 3>(a, grid, stream, tb, delta, finish, w);
}

// Whether the edges of a block-diagonal with `blocks` blocks over all chains
// go by rows (16 launches) rather than by anti-diagonals (30 or 31).
bool row_edges(int64_t blocks) { return blocks >= kRowMinBlocks; }

void launch_edge_row(int a, int blocks, hipStream_t stream, const Tables &tb, int delta, int finish, const Work &w)
{
    const unsigned chunks = (unsigned)((tb.M + kEdgeThreads * kRowBudgets) / (kEdgeThreads * kRowBudgets));
    const dim3 grid(chunks, blocks, tb.n_chains);
    switch (a / 4) {
    case 0:
        launch_edge_row_0(a, grid, stream, tb, delta, finish, w);
        break;
    case 1:
        launch_edge_row_1(a, grid, stream, tb, delta, finish, w);
        break;
    case 2:
        launch_edge_row_2(a, grid, stream, tb, delta, finish, w);
        break;
    default:
        launch_edge_row_3(a, grid, stream, tb, delta, finish, w);
        break;
    }
}

}  // namespace rotor
