"""MI355X (gfx950) prefix-cache-aware router: batched longest-prefix match of
requests against every peer's radix-tree estimate, with the argmax over peers
and anti-entropy tree updates, behind the C ABI in include/prefix_router.h."""
from .router import (Forest, RouterError, pr_forest_check, pr_forest_create,  # noqa: F401
                     pr_forest_destroy, pr_forest_host_image, pr_forest_info_get, pr_last_error,
                     pr_load_snapshot, pr_load_snapshot_device, pr_export_snapshot, pr_merge, pr_route,
                     pr_route_noalloc, pr_route_select, pr_tree_tokens, pr_forest_compact, pr_set_local_peer, pr_set_time, pr_touch, pr_evict_lru, eligible_words,
                     PR_SELECT_PREFER_LOCAL)
