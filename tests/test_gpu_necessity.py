"""Static reclamation OOMs on a prefill-sized activation burst; the dynamic
toggle runs it clean; a recommit needs the caching allocator's memory back
first (the paper, Section 4)."""
import pytest
import torch

from paper_2608_23658_amd import necessity
from tests.gpu_helpers import require_gpu, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def test_static_commit_ooms_dynamic_toggle_runs_the_burst():
    say("necessity demo: fill device memory, 3 GiB reserve over 32 layers")
    r = necessity.run()
    say(r)
    assert r["static_burst_oom"] is True
    assert r["dynamic_burst_ok"] is True
    assert r["recommit_without_empty_cache"] == "oom"
    assert r["pool_consistent_after_failed_commit"] is True
    assert r["recommit_ok"] is True
    free, total = torch.cuda.mem_get_info()
    assert free > total // 2          # everything was released
