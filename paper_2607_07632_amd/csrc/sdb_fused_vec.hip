// Instances of the fused pass: 4-row items (128-bit loads), launch bound kMaxBlock.

#include "sdb_fused.h"

namespace sdb {

const void* pick_fused_vec(int ipt, int terminal) {
    if (ipt == 1) { SDB_FUSED_TERMINALS(4, 1, false, kMaxBlock, 0) }
    if (ipt == 2) { SDB_FUSED_TERMINALS(4, 2, false, kMaxBlock, 0) }
    if (ipt == 4) { SDB_FUSED_TERMINALS(4, 4, false, kMaxBlock, 0) }
    return nullptr;
}

}  // namespace sdb
