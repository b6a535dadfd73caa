"""Host-side scheduling layer above the layer step: an iteration-latency
predictor fitted to measured steps, and the SLO slack accounting and
discrete-event simulator of prefill/decode multiplexing built on it."""
from .predictor import LatencyModel, batch_features, FEATURES  # noqa: F401
from .slo import SLO, Request, admits_chunk, attainment  # noqa: F401
from .sim import Cluster, Simulator, attainment_sweep, light_load_slo, per_request_ttft, synthetic_requests  # noqa: F401
