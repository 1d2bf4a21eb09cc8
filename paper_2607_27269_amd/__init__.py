"""MI355X-native functional-reconstruction step for converted MLA attention layers."""
from . import configs  # noqa: F401
