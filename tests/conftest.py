import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


# The GPU tests write up to a few GB of checkpoints under pytest's temporary
# directory; where the disk holding /tmp is nearly full, they use /dev/shm.
_MIN_TMP_FREE = 8 << 30


def _free(path):
    try:
        import shutil

        return shutil.disk_usage(path).free
    except OSError:
        return 0


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU")
    config.addinivalue_line("markers", "slow: long-running CPU test")
    if (not config.option.basetemp and _free("/tmp") < _MIN_TMP_FREE
            and _free("/dev/shm") >= 2 * _MIN_TMP_FREE):
        config.option.basetemp = f"/dev/shm/sllm_pytest_{os.getuid()}"


@pytest.fixture(scope="session")
def gpu_device():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda", 0)
