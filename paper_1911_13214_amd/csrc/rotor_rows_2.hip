// Row edges with 8 to 11 low splits (see rotor_rows.h).
#include "rotor_rows.h"

namespace rotor {

void launch_edge_row_2(int a, dim3 grid, hipStream_t stream, const Tables &tb, int delta, int finish, const Work &w)
{
    launch_edge_row_range<8, 11>(a, grid, stream, tb, delta, finish, w);
}

}  // namespace rotor
