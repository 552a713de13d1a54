import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


import pytest  # noqa: E402


def _say(config, msg):
    """Write msg to the terminal's stderr with pytest's output capture
    suspended (fd-level capture would otherwise hold it back until a
    failure)."""
    capman = config.pluginmanager.getplugin("capturemanager")
    if capman is None:
        sys.stderr.write(msg + "\n")
        sys.stderr.flush()
        return
    with capman.global_and_fixture_disabled():
        sys.stderr.write(msg + "\n")
        sys.stderr.flush()


@pytest.fixture(autouse=True)
def _announce_gpu_case(request):
    """Name every GPU test on the real stderr before it touches the device,
    so a run that ends abruptly still shows which case was running."""
    if request.node.get_closest_marker("gpu") is not None:
        _say(request.config, f"[gpu-case] {request.node.nodeid}")
    yield


@pytest.fixture
def report(request):
    """report(msg): a line in the test log, passing runs included."""
    return lambda msg: _say(request.config, msg)


_STEPS = {}


@pytest.fixture(scope="session")
def step_cache():
    """Synthetic decode steps shared by the tests of one session."""
    import synth

    def get(name, seed=0, with_weight=True):
        key = (name, seed, with_weight)
        if key not in _STEPS:
            _STEPS[key] = synth.make_step(name, seed, with_weight=with_weight)
        return _STEPS[key]
    return get
