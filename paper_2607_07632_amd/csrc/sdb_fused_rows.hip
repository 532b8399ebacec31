// Instances of the fused pass: 1-row items (columns not 16-byte aligned).

#include "sdb_fused.h"

namespace sdb {

const void* pick_fused_rows(int ipt, int terminal) {
    if (ipt == 1) { SDB_FUSED_TERMINALS(1, 1, false, kMaxBlock, 0) }
    if (ipt == 2) { SDB_FUSED_TERMINALS(1, 2, false, kMaxBlock, 0) }
    if (ipt == 4) { SDB_FUSED_TERMINALS(1, 4, false, kMaxBlock, 0) }
    return nullptr;
}

}  // namespace sdb
