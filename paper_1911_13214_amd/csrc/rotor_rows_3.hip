// Row edges with 12 to 15 low splits (see rotor_rows.h).
#include "rotor_rows.h"

namespace rotor {

void launch_edge_row_3(int a, dim3 grid, hipStream_t stream, const Tables &tb, int delta, int finish, const Work &w)
{
    launch_edge_row_range<12, 15>(a, grid, stream, tb, delta, finish, w);
}

}  // namespace rotor
