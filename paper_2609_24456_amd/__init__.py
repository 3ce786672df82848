"""MI355X-native experience path (ingest, priority update, sampling,
gather/transform, GAE, minibatch shuffle-gather) behind the C ABI of
libconduit.so; ``conduit`` is its Python binding."""
from . import conduit  # noqa: F401
