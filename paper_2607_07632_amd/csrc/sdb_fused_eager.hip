// Instances of the fused pass: 4-row items with eager column loads.

#include "sdb_fused.h"

namespace sdb {

const void* pick_fused_eager(int ipt, int terminal) {
    if (ipt == 1) { SDB_FUSED_TERMINALS(4, 1, true, kMaxBlock, 0) }
    if (ipt == 2) { SDB_FUSED_TERMINALS(4, 2, true, kMaxBlock, 0) }
    return nullptr;
}

}  // namespace sdb
